"""Cost model pinned to the paper's printed figures; DN-table structure."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2609_10018_amd import cost, inputs
from paper_2609_10018_amd.inputs import CONFIGS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_pins.json")


def test_base_flops_match_table1():
    pins = json.load(open(GOLDEN))
    cfg = CONFIGS["vit_b"]
    table = inputs.make_dn_table(cfg)
    g = cost.paper_macs(cfg, table, 0) / 1e9
    assert abs(g - pins["vit_b_base_gflops"]["value"]) < 0.02


def test_param_count_matches_table3():
    pins = json.load(open(GOLDEN))
    n = inputs.param_count(CONFIGS["vit_b"])
    assert n == 86_567_656
    assert abs(n * 4 / 2 ** 20 - pins["vit_b_size_mb"]["value"]) < 0.1


@pytest.mark.parametrize("name", list(CONFIGS))
def test_flops_monotone_and_equal_direct_count(name):
    cfg = CONFIGS[name]
    table = inputs.make_dn_table(cfg)
    w = inputs.make_weights(cfg) if name not in ("vit_b", "vit_b_emb") else None
    prev = None
    for k in range(table.num_modes):
        f = cost.flops_per_image(cfg, table, k)
        if prev is not None:
            assert f <= prev
        prev = f
        if w is None:
            continue
        p = oracle.extract_dense(w, cfg, table, k)
        T, N = cfg.tokens, cfg.num_patches
        direct = 2 * N * p["patch_w"].size
        for lp in p["layers"]:
            h = lp["qkv_w"].shape[0] // (3 * cfg.head_dim)
            direct += 2 * T * (lp["qkv_w"].size + lp["proj_w"].size +
                               lp["fc1_w"].size + lp["fc2_w"].size)
            direct += 2 * 2 * T * T * cfg.head_dim * h
        direct += 2 * p["head_w"].size
        assert f == pytest.approx(direct, rel=1e-12)


def test_headline_flops_per_image():
    cfg = CONFIGS["vit_b"]
    table = inputs.make_dn_table(cfg)
    got = [cost.flops_per_image(cfg, table, k) / 1e9 for k in range(5)]
    np.testing.assert_allclose(got, [35.128, 26.404, 17.680, 8.957, 5.671], atol=2e-3)


@pytest.mark.parametrize("name", list(CONFIGS))
def test_dn_tables_nested_and_in_range(name):
    cfg = CONFIGS[name]
    t = inputs.make_dn_table(cfg)
    assert t.n_heads.shape == (len(inputs.MODE_CAPS[name]), cfg.depth)
    assert (t.n_heads >= 1).all() and (t.n_heads <= cfg.heads).all()
    assert (t.n_mlp >= 1).all() and (t.n_mlp <= cfg.mlp_hidden).all()
    assert (np.diff(t.n_heads, axis=0) <= 0).all() and (np.diff(t.n_mlp, axis=0) <= 0).all()
    assert (t.n_heads[0] == cfg.heads).all() and (t.n_mlp[0] == cfg.mlp_hidden).all()
    for l in range(cfg.depth):
        assert sorted(t.head_order[l]) == list(range(cfg.heads))
        assert sorted(t.mlp_order[l]) == list(range(cfg.mlp_hidden))
    assert sorted(t.embed_order) == list(range(cfg.dim))
    assert t.n_embed.shape == (t.num_modes,) and t.n_embed[0] == cfg.dim
    assert (np.diff(t.n_embed) <= 0).all() and (t.n_embed >= 1).all()
    if cfg.dtype == inputs.BF16:
        assert (t.n_embed % 8 == 0).all()


def test_vit_s_layer_ratios_give_layer_dependent_widths():
    cfg = CONFIGS["vit_s"]
    t = inputs.make_dn_table(cfg)
    r = inputs.layer_ratios(cfg)
    assert ((r >= 0.15) & (r <= 1.0)).all()
    assert len(set(t.n_mlp[1].tolist())) > 1
    caps = inputs.MODE_CAPS["vit_s"]
    for k in range(1, 5):
        for l in range(cfg.depth):
            assert t.n_heads[k, l] == max(1, int(np.floor(caps[k][0] * r[l] + 0.5)))
            assert t.n_mlp[k, l] == max(1, int(np.floor(caps[k][1] * r[l] + 0.5)))


def test_bf16_round_is_rne():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 3.0e38,
                  np.inf, -np.inf, 0.0], dtype=np.float32)
    got = inputs.bf16_round(x)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa is 1.
    ref = np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5, 2.9975e38, np.inf, -np.inf, 0.0],
                   dtype=np.float32)
    np.testing.assert_array_equal(got[[0, 1, 2, 3, 4, 6, 7, 8]], ref[[0, 1, 2, 3, 4, 6, 7, 8]])
    assert np.isnan(inputs.bf16_round(np.array([np.nan], dtype=np.float32)))[0]
    y = np.random.default_rng(0).standard_normal(1000).astype(np.float32)
    r = inputs.bf16_round(y)
    assert (r.view(np.uint32) & 0xFFFF == 0).all()
    assert np.max(np.abs(r - y) / np.abs(y)) <= 2 ** -8
