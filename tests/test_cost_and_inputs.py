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


@pytest.mark.parametrize("name", ["tiny", "tiny_emb", "vit_ti"])
def test_channel_orders_follow_l1_saliency(name):
    """Eq. 4's saliency, written out with loops: a head's score is the mean
    |w| over its q, k and v rows, a unit's the mean |w| of its fc1 row, an
    embedding channel's the mean |w| of its patch-embedding row; the order
    lists them by descending score (equal scores: lower index first)."""
    cfg = CONFIGS[name]
    w = inputs.make_weights(cfg)
    t = inputs.make_dn_table(cfg)
    d, hd = cfg.dim, cfg.head_dim

    def mean_abs(rows):
        tot, n = 0.0, 0
        for r in rows:
            for v in np.asarray(r, dtype=np.float64).reshape(-1):
                tot += abs(float(v))
                n += 1
        return tot / n

    def check(order, scores):
        assert sorted(order.tolist()) == list(range(len(scores)))
        for a, b in zip(order[:-1], order[1:]):
            assert scores[a] > scores[b] or (scores[a] == scores[b] and a < b)

    for l in range(cfg.depth):
        hs = [mean_abs([w["qkv_w"][l][q * d + i * hd + c] for q in range(3) for c in range(hd)])
              for i in range(cfg.heads)]
        check(t.head_order[l], hs)
        us = [mean_abs([w["fc1_w"][l][j]]) for j in range(cfg.mlp_hidden)]
        check(t.mlp_order[l], us)
    es = [mean_abs([w["patch_w"][c]]) for c in range(d)]
    check(t.embed_order, es)


def test_saliency_order_ties_and_explicit_weights():
    rows = np.array([[1.0, -1.0], [2.0, 0.0], [0.5, 0.5], [-3.0, 1.0], [0.0, 2.0]])
    # scores 1, 1, 0.5, 2, 1: descending, equal scores by index
    assert inputs.saliency_order(rows).tolist() == [3, 0, 1, 4, 2]
    # Reversing layer 0's units (fc1 rows) reverses the index of every score,
    # so the order maps j -> m - 1 - j; other layers keep theirs.
    cfg = CONFIGS["tiny"]
    w = inputs.make_weights(cfg)
    w2 = {k: np.array(v, copy=True) for k, v in w.items()}
    w2["fc1_w"][0] = w2["fc1_w"][0][::-1].copy()
    t, t2 = inputs.make_dn_table(cfg), inputs.make_dn_table(cfg, w2)
    m = cfg.mlp_hidden
    assert np.unique(np.abs(w["fc1_w"][0]).mean(axis=1)).size == m
    np.testing.assert_array_equal(t2.mlp_order[0], m - 1 - t.mlp_order[0])
    np.testing.assert_array_equal(t2.mlp_order[1:], t.mlp_order[1:])
    np.testing.assert_array_equal(t2.head_order, t.head_order)


@pytest.mark.parametrize("name", ["tiny", "vit_ti", "vit_ti_emb"])
def test_dense_model_bytes_count_the_extracted_model(name):
    """cost.dense_model_bytes equals the sizes of the oracle's extracted
    dense model (F3), matrices at 2 bytes and everything else at 4."""
    cfg = CONFIGS[name]
    w = inputs.make_weights(cfg)
    t = inputs.make_dn_table(cfg)
    mats = set(inputs.MATRIX_KEYS)
    for k in range(t.num_modes):
        p = oracle.extract_dense(w, cfg, t, k)
        total = 0
        for key, v in p.items():
            if key == "layers":
                for lp in v:
                    total += sum(a.size * (2 if kk in mats else 4) for kk, a in lp.items())
            elif isinstance(v, np.ndarray):
                total += v.size * (2 if key in mats else 4)
        assert cost.dense_model_bytes(cfg, t, k) == total, (name, k)


def test_growth_step_flops_decomposition():
    """The growth step's count = forward + head backward + activation
    gradients (the forward's layer contractions once more) + attention
    backward (2.5x the forward's QK^T and PV) + weight gradients of the
    re-introduced slices: none when mode k + 1 equals mode k, all of the
    layer contractions once more when mode k + 1 keeps nothing."""
    from types import SimpleNamespace
    cfg = inputs.CONFIGS["vit_b"]
    L = cfg.depth
    h0, m0 = np.full(L, cfg.heads), np.full(L, cfg.mlp_hidden)
    f = cost.gemm_flops(cfg, SimpleNamespace(n_heads=[h0], n_mlp=[m0]), 0)
    layers = f["qkv"] + f["proj"] + f["fc1"] + f["fc2"]
    base = sum(f.values()) + 2.0 * cfg.dim * cfg.num_classes + layers + 2.5 * f["attn"]
    same = SimpleNamespace(n_heads=[h0, h0], n_mlp=[m0, m0])
    none = SimpleNamespace(n_heads=[h0, 0 * h0], n_mlp=[m0, 0 * m0])
    assert cost.growth_step_flops(cfg, same, 0) == pytest.approx(base, rel=1e-12)
    assert cost.growth_step_flops(cfg, none, 0) == pytest.approx(base + layers, rel=1e-12)
    t = inputs.make_dn_table(cfg)
    assert (cost.growth_step_flops(cfg, same, 0) < cost.growth_step_flops(cfg, t, 0)
            < cost.growth_step_flops(cfg, none, 0))
