"""Pins of the fp64 oracle against things other than itself (CPU only).

* brute-force per-element loops for attention, LayerNorm, GELU, patchify;
* closed forms (GELU at known points, LayerNorm moments, softmax row sums);
* a textbook ViT from torch fp64 library ops (full width, and pruned modes
  with masks built one head / unit at a time);
* mask form (F2) vs gather form (F3 + F1) for every mode of every config;
* permutation invariance, bias-mask irrelevance and locality.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2609_10018_amd import inputs
from paper_2609_10018_amd.inputs import CONFIGS, DNTable, ModelConfig
from textbook import loop_extract_embed, loop_masked_weights, rel_err, torch_vit

MINI = ModelConfig("mini", 48, 8, 3, 96, 3, 3, 192, 7, inputs.FP32, 3)


def mini_table(cfg=MINI):
    rng = np.random.default_rng(11)
    L = cfg.depth
    n_heads = np.array([[3] * L, [2, 3, 1], [1, 1, 1]], dtype=np.int32)
    n_mlp = np.array([[192] * L, [100, 57, 150], [1, 13, 64]], dtype=np.int32)
    ho = np.stack([rng.permutation(cfg.heads) for _ in range(L)]).astype(np.int32)
    mo = np.stack([rng.permutation(cfg.mlp_hidden) for _ in range(L)]).astype(np.int32)
    return DNTable(n_heads, n_mlp, ho, mo)


@pytest.fixture(scope="module")
def mini():
    w = inputs.make_weights(MINI)
    x = inputs.make_images(MINI, 3)
    return w, x, mini_table()


# ---------------------------------------------------------------- brute force

def test_patchify_matches_index_loop():
    rng = np.random.default_rng(5)
    img = rng.standard_normal((2, 3, 12, 12))
    P = 4
    got = oracle.patchify(img, P)
    for b in range(2):
        for py in range(3):
            for px in range(3):
                n = py * 3 + px
                f = 0
                for c in range(3):
                    for i in range(P):
                        for j in range(P):
                            assert got[b, n, f] == img[b, c, py * P + i, px * P + j]
                            f += 1


def test_layer_norm_loop_and_moments():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((5, 24)) * 3.0 + 1.5
    g = rng.standard_normal(24)
    b = rng.standard_normal(24)
    eps = 1e-6
    got = oracle.layer_norm(x, g, b, eps)
    for r in range(5):
        mu = sum(x[r]) / 24
        var = sum((v - mu) ** 2 for v in x[r]) / 24
        for c in range(24):
            ref = (x[r, c] - mu) / math.sqrt(var + eps) * g[c] + b[c]
            assert abs(got[r, c] - ref) < 1e-12 * max(1.0, abs(ref))
    plain = oracle.layer_norm(x, np.ones(24), np.zeros(24), eps)
    var = x.var(axis=-1)
    np.testing.assert_allclose(plain.mean(axis=-1), 0.0, atol=1e-13)
    np.testing.assert_allclose((plain ** 2).mean(axis=-1), var / (var + eps), rtol=1e-12)


def test_gelu_closed_forms():
    # Phi(1) = 0.8413447460685429..., Phi(-1) = 1 - Phi(1), GELU(0) = 0.
    z = np.array([0.0, 1.0, -1.0, 2.0, -3.0])
    got = oracle.gelu(z)
    ref = np.array([0.0, 0.8413447460685429, -0.15865525393145707,
                    2 * 0.9772498680518208, -3 * 0.0013498980316301])
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-15)
    zz = np.linspace(-6, 6, 101)
    ref2 = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in zz])
    np.testing.assert_allclose(oracle.gelu(zz), ref2, rtol=1e-14, atol=1e-16)


def test_softmax_loop_and_row_sums():
    rng = np.random.default_rng(7)
    s = rng.standard_normal((4, 9)) * 5
    p = oracle.softmax_rows(s)
    for r in range(4):
        den = sum(math.exp(v) for v in s[r])
        for c in range(9):
            assert abs(p[r, c] - math.exp(s[r, c]) / den) < 1e-14
    np.testing.assert_allclose(p.sum(axis=-1), 1.0, atol=1e-12)
    big = oracle.softmax_rows(np.array([[1000.0, 999.0, -1000.0]]))
    assert np.isfinite(big).all()


def test_attention_matches_per_element_loop():
    rng = np.random.default_rng(8)
    B, T, d, h, hd = 2, 5, 6, 2, 3
    u = rng.standard_normal((B, T, d))
    qkv_w = rng.standard_normal((3 * h * hd, d))
    qkv_b = rng.standard_normal(3 * h * hd)
    got = oracle.attention(u, qkv_w, qkv_b, hd)
    for b in range(B):
        lin = [[sum(u[b, t, c] * qkv_w[r, c] for c in range(d)) + qkv_b[r]
                for r in range(3 * h * hd)] for t in range(T)]
        for i in range(h):
            q = lambda t, c: lin[t][i * hd + c]
            k = lambda t, c: lin[t][h * hd + i * hd + c]
            v = lambda t, c: lin[t][2 * h * hd + i * hd + c]
            for t in range(T):
                s = [sum(q(t, c) * k(j, c) for c in range(hd)) / math.sqrt(hd) for j in range(T)]
                mx = max(s)
                e = [math.exp(x - mx) for x in s]
                den = sum(e)
                for c in range(hd):
                    ref = sum(e[j] / den * v(j, c) for j in range(T))
                    assert abs(got[b, t, i * hd + c] - ref) < 1e-12 * max(1.0, abs(ref))


# ---------------------------------------------------------- textbook ViT (I1)

@pytest.mark.parametrize("cfg", [CONFIGS["tiny"], MINI], ids=["tiny", "mini"])
def test_full_width_equals_textbook_vit(cfg):
    w = inputs.make_weights(cfg)
    x = inputs.make_images(cfg, 3)
    got = oracle.vit_forward(oracle.canonical_params(w, cfg.depth), x,
                             cfg.dim // cfg.heads, cfg.ln_eps)
    ref = torch_vit(w, x, cfg)
    assert rel_err(got, ref) < 1e-10


def test_full_width_vit_ti_equals_textbook():
    cfg = CONFIGS["vit_ti"]
    w = inputs.make_weights(cfg)
    x = inputs.make_images(cfg, 1)
    got = oracle.vit_forward(oracle.canonical_params(w, cfg.depth), x, cfg.head_dim, cfg.ln_eps)
    assert rel_err(got, torch_vit(w, x, cfg)) < 1e-10


def test_pruned_modes_equal_textbook_on_loop_masked_weights(mini):
    w, x, table = mini
    for k in range(table.num_modes):
        ref = torch_vit(loop_masked_weights(w, MINI, table, k), x, MINI)
        got = oracle.elastic_forward(w, MINI, table, k, x)
        assert rel_err(got, ref) < 1e-10, k


def test_tiny_modes_equal_textbook_on_loop_masked_weights():
    cfg = CONFIGS["tiny"]
    w = inputs.make_weights(cfg)
    x = inputs.make_images(cfg, cfg.batch)
    table = inputs.make_dn_table(cfg)
    for k in range(table.num_modes):
        ref = torch_vit(loop_masked_weights(w, cfg, table, k), x, cfg)
        assert rel_err(oracle.elastic_forward(w, cfg, table, k, x), ref) < 1e-10


# ------------------------------------------------------- C1 / C2 self-checks

def test_c1_full_width_mask_equals_unmasked(mini):
    w, x, table = mini
    f1 = oracle.vit_forward(oracle.canonical_params(w, MINI.depth), x, 32, MINI.ln_eps)
    f2 = oracle.elastic_forward_masked(w, MINI, table, 0, x)
    assert rel_err(f2, f1) < 1e-12


@pytest.mark.parametrize("name", ["tiny", "vit_ti", "vit_s", "vit_b"])
def test_c2_mask_form_equals_gather_form(name):
    cfg = CONFIGS[name]
    w = inputs.make_weights(cfg)
    table = inputs.make_dn_table(cfg)
    nimg = {"tiny": 4, "vit_ti": 2, "vit_s": 1, "vit_b": 1}[name]
    x = inputs.make_images(cfg, nimg)
    for k in range(table.num_modes):
        f2 = oracle.elastic_forward_masked(w, cfg, table, k, x)
        f13 = oracle.elastic_forward(w, cfg, table, k, x)
        assert rel_err(f13, f2) < 1e-10, (name, k)


def test_c2_mini_all_modes(mini):
    w, x, table = mini
    for k in range(table.num_modes):
        f2 = oracle.elastic_forward_masked(w, MINI, table, k, x)
        f13 = oracle.elastic_forward(w, MINI, table, k, x)
        assert rel_err(f13, f2) < 1e-10


# ------------------------------------------------------------- invariants

def test_i2_permutation_invariance(mini):
    w, x, _ = mini
    hd = MINI.dim // MINI.heads
    base = oracle.vit_forward(oracle.canonical_params(w, MINI.depth), x, hd, MINI.ln_eps)
    rng = np.random.default_rng(12)
    p = oracle.canonical_params(w, MINI.depth)
    for lp in p["layers"]:
        hp = rng.permutation(MINI.heads)
        chans = np.concatenate([np.arange(i * hd, (i + 1) * hd) for i in hp])
        rows = np.concatenate([chans, MINI.dim + chans, 2 * MINI.dim + chans])
        lp["qkv_w"], lp["qkv_b"] = lp["qkv_w"][rows], lp["qkv_b"][rows]
        lp["proj_w"] = lp["proj_w"][:, chans]
        up = rng.permutation(MINI.mlp_hidden)
        lp["fc1_w"], lp["fc1_b"] = lp["fc1_w"][up], lp["fc1_b"][up]
        lp["fc2_w"] = lp["fc2_w"][:, up]
    got = oracle.vit_forward(p, x, hd, MINI.ln_eps)
    assert rel_err(got, base) < 1e-12


def test_i3_bias_masks_irrelevant(mini):
    w, x, table = mini
    for k in range(table.num_modes):
        a = oracle.elastic_forward_masked(w, MINI, table, k, x, mask_biases=True)
        b = oracle.elastic_forward_masked(w, MINI, table, k, x, mask_biases=False)
        assert rel_err(a, b) < 1e-12


def test_i4_locality(mini):
    w, x, table = mini
    k = 2
    w2 = {key: np.array(v, copy=True) for key, v in w.items()}
    rng = np.random.default_rng(13)
    hd = MINI.dim // MINI.heads
    for l in range(MINI.depth):
        act_h, act_m = oracle.active_sets(table, k, l)
        off_h = sorted(set(range(MINI.heads)) - set(act_h.tolist()))
        off_m = sorted(set(range(MINI.mlp_hidden)) - set(act_m.tolist()))
        for i in off_h:
            for t in range(3):
                sl = slice(t * MINI.dim + i * hd, t * MINI.dim + (i + 1) * hd)
                w2["qkv_w"][l][sl] = rng.standard_normal((hd, MINI.dim))
                w2["qkv_b"][l][sl] = rng.standard_normal(hd)
            w2["proj_w"][l][:, i * hd:(i + 1) * hd] = rng.standard_normal((MINI.dim, hd))
        for j in off_m:
            w2["fc1_w"][l][j] = rng.standard_normal(MINI.dim)
            w2["fc1_b"][l][j] = rng.standard_normal()
            w2["fc2_w"][l][:, j] = rng.standard_normal(MINI.dim)
    a = oracle.elastic_forward(w, MINI, table, k, x)
    b = oracle.elastic_forward(w2, MINI, table, k, x)
    assert np.array_equal(a, b)
    a2 = oracle.elastic_forward_masked(w, MINI, table, k, x)
    b2 = oracle.elastic_forward_masked(w2, MINI, table, k, x)
    assert np.array_equal(a2, b2)


# ------------------------------------------------- narrower embedding (E1-E4)

def test_masked_layer_norm_is_layer_norm_of_the_active_channels():
    rng = np.random.default_rng(21)
    x = rng.standard_normal((5, 40)) * 3 + 1
    g, b = rng.standard_normal(40), rng.standard_normal(40)
    act = np.sort(rng.permutation(40)[:17])
    m = np.zeros(40)
    m[act] = 1.0
    got = oracle.layer_norm_masked(x, g * m, b * m, 1e-6, m)
    ref = oracle.layer_norm(x[:, act], g[act], b[act], 1e-6)
    np.testing.assert_allclose(got[:, act], ref, rtol=1e-13, atol=1e-13)
    assert np.all(got[:, np.setdiff1d(np.arange(40), act)] == 0.0)
    full = oracle.layer_norm_masked(x, g, b, 1e-6, np.ones(40))
    np.testing.assert_allclose(full, oracle.layer_norm(x, g, b, 1e-6), rtol=1e-13, atol=1e-13)


def test_embed_modes_equal_textbook_on_extracted_channels():
    """Every tiny_emb mode: the textbook ViT (F.layer_norm over the d_k
    channels it is given) on weights copied channel by channel equals both the
    mask form and the gather form."""
    import dataclasses
    cfg = CONFIGS["tiny_emb"]
    w = inputs.make_weights(cfg)
    x = inputs.make_images(cfg, cfg.batch)
    table = inputs.make_dn_table(cfg)
    assert list(table.n_embed) == [64, 48, 24]
    for k in range(table.num_modes):
        sub, E = loop_extract_embed(w, cfg, table, k)
        ref = torch_vit(sub, x, dataclasses.replace(cfg, dim=E), head_dim=cfg.head_dim)
        assert rel_err(oracle.elastic_forward(w, cfg, table, k, x), ref) < 1e-10, k
        assert rel_err(oracle.elastic_forward_masked(w, cfg, table, k, x), ref) < 1e-10, k


@pytest.mark.parametrize("name", ["vit_ti_emb", "vit_b_emb"])
def test_c2_embed_mask_form_equals_gather_form(name):
    cfg = CONFIGS[name]
    w = inputs.make_weights(cfg)
    table = inputs.make_dn_table(cfg)
    x = inputs.make_images(cfg, 1)
    for k in range(1, table.num_modes):
        assert table.n_embed[k] < cfg.dim
        f2 = oracle.elastic_forward_masked(w, cfg, table, k, x)
        f13 = oracle.elastic_forward(w, cfg, table, k, x)
        assert rel_err(f13, f2) < 1e-10, (name, k)


def test_i4_embed_locality():
    """Weights of the embedding channels a mode drops do not change its logits."""
    cfg = CONFIGS["tiny_emb"]
    w = inputs.make_weights(cfg)
    x = inputs.make_images(cfg, 2)
    table = inputs.make_dn_table(cfg)
    k = 2
    off = np.setdiff1d(np.arange(cfg.dim), oracle.active_embed(table, k, cfg.dim))
    rng = np.random.default_rng(22)
    w2 = {key: np.array(v, copy=True) for key, v in w.items()}
    w2["patch_w"][off] = rng.standard_normal(w2["patch_w"][off].shape)
    for key in ("patch_b", "cls", "norm_g", "norm_b"):
        w2[key][off] = 7.0
    w2["pos"][:, off] = -3.0
    w2["head_w"][:, off] = 5.0
    for key in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "proj_b", "fc2_b"):
        w2[key][:, off] = 9.0
    w2["qkv_w"][:, :, off] = 4.0
    w2["fc1_w"][:, :, off] = -4.0
    w2["proj_w"][:, off, :] = 2.0
    w2["fc2_w"][:, off, :] = 2.0
    a = oracle.elastic_forward(w, cfg, table, k, x)
    b = oracle.elastic_forward(w2, cfg, table, k, x)
    assert np.array_equal(a, b)
    am = oracle.elastic_forward_masked(w, cfg, table, k, x)
    bm = oracle.elastic_forward_masked(w2, cfg, table, k, x)
    assert rel_err(bm, am) < 1e-12
    # and they do change a mode that keeps every channel
    assert not np.array_equal(oracle.elastic_forward(w, cfg, table, 0, x),
                              oracle.elastic_forward(w2, cfg, table, 0, x))
