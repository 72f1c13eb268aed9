"""Pins of the growth-step oracle (oracle/growth.py) against what the paper
and the mathematics fix, independent of the oracle's own arithmetic:

* its forward and loss equal the pinned inference oracle's logits through a
  plain cross-entropy;
* its gradient equals central finite differences of the loss, and torch fp64
  autograd through the textbook ViT (mask form of the DN, Eqs. 4 and 6);
* Eq. 9's mask is exactly (mode k's weights) - (mode k+1's weights), built
  here from the brute-force per-head / per-unit masking;
* the update leaves mode k+1's logits bit-identical (its weights are frozen)
  and moves only masked entries; norm clipping bounds the step;
* planted mistakes in the backward fail these pins.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import growth as og
from paper_2609_10018_amd import inputs
from paper_2609_10018_amd.inputs import CONFIGS
from test_oracle import MINI, mini_table
from textbook import loop_masked_weights, rel_err, torch_vit


def _labels(cfg, B, seed=3):
    return np.random.default_rng(seed).integers(0, cfg.num_classes, size=B)


@pytest.fixture(scope="module")
def mini():
    w = {k: np.asarray(v, dtype=np.float64) for k, v in inputs.make_weights(MINI).items()}
    x = inputs.make_images(MINI, 2)
    return w, x, mini_table(), _labels(MINI, 2)


def _masks(cfg, table, k):
    """Brute-force {0,1} masks of mode k's weights (loop over heads / units)."""
    ones = {key: np.ones(shp) for key, shp in og._canonical_shapes(cfg).items()}
    m = loop_masked_weights(ones, cfg, table, k)
    d, hd = cfg.dim, cfg.dim // cfg.heads
    for l in range(cfg.depth):                     # biases follow their rows
        m["qkv_b"][l] = m["qkv_w"][l][:, 0]
        m["fc1_b"][l] = m["fc1_w"][l][:, 0]
    return m


@pytest.mark.parametrize("k", [0, 1, 2])
def test_loss_equals_cross_entropy_of_inference_logits(mini, k):
    w, x, t, y = mini
    loss, _ = og.loss_and_grad(w, MINI, t, k, x, y)
    logits = oracle.elastic_forward_masked(w, MINI, t, k, x)
    ref = F.cross_entropy(torch.as_tensor(logits), torch.as_tensor(y)).item()
    assert abs(loss - ref) < 1e-12 * max(1.0, abs(ref))


@pytest.mark.parametrize("k", [0, 1])
def test_gradient_matches_central_differences(mini, k):
    w, x, t, y = mini
    _, grad = og.loss_and_grad(w, MINI, t, k, x, y)
    active = _masks(MINI, t, k)
    rng = np.random.default_rng(7 + k)
    checked = 0
    for key in sorted(grad):
        m = active.get(key) if key in ("qkv_w", "qkv_b", "proj_w", "fc1_w", "fc1_b", "fc2_w") \
            else None
        flat = np.flatnonzero(m.reshape(-1)) if m is not None else np.arange(w[key].size)
        for idx in rng.choice(flat, size=min(3, flat.size), replace=False):
            wp = dict(w)
            h = 1e-5 * max(1.0, abs(w[key].reshape(-1)[idx]))
            a = w[key].copy().reshape(-1)
            a[idx] += h
            wp[key] = a.reshape(w[key].shape)
            lp, _ = og.loss_and_grad(wp, MINI, t, k, x, y)
            a[idx] -= 2 * h
            wp[key] = a.reshape(w[key].shape)
            lm, _ = og.loss_and_grad(wp, MINI, t, k, x, y)
            fd = (lp - lm) / (2 * h)
            g = grad[key].reshape(-1)[idx]
            assert abs(fd - g) <= 1e-6 * max(1e-3, abs(g)) + 1e-9, (key, idx, fd, g)
            checked += 1
    assert checked >= 3 * len(grad) - 3


@pytest.mark.parametrize("k", [0, 1, 2])
def test_gradient_matches_torch_autograd(mini, k):
    """Textbook ViT on M (.) W (masks inside the graph), F.cross_entropy,
    autograd: the gradient with respect to W is the oracle's canonical one."""
    w, x, t, y = mini
    _, grad = og.loss_and_grad(w, MINI, t, k, x, y)
    masks = _masks(MINI, t, k)
    leaves = {key: torch.tensor(v, dtype=torch.float64, requires_grad=True) for key, v in w.items()}
    eff = {key: (leaves[key] * torch.as_tensor(masks[key]) if key in
                 ("qkv_w", "qkv_b", "proj_w", "fc1_w", "fc1_b", "fc2_w") else leaves[key])
           for key in leaves}
    logits = torch_vit(eff, x, MINI, grad=True)
    F.cross_entropy(logits, torch.as_tensor(y)).backward()
    for key in grad:
        ref = leaves[key].grad.numpy()
        assert np.max(np.abs(grad[key] - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref))), key


@pytest.mark.parametrize("k", [0, 1])
def test_mask_is_mode_k_minus_mode_k_plus_1(mini, k):
    _, _, t, _ = mini
    G = og.growth_mask(MINI, t, k)
    mk, mp = _masks(MINI, t, k), _masks(MINI, t, k + 1)
    for key in G:
        if key in ("qkv_w", "qkv_b", "proj_w", "fc1_w", "fc1_b", "fc2_w"):
            np.testing.assert_array_equal(G[key], mk[key] - mp[key])
        else:
            assert not G[key].any(), key        # LayerNorm, embeddings, head, proj/fc2 bias
    hd, d = MINI.dim // MINI.heads, MINI.dim
    for l in range(MINI.depth):
        dh = int(t.n_heads[k][l] - t.n_heads[k + 1][l])
        dm = int(t.n_mlp[k][l] - t.n_mlp[k + 1][l])
        assert G["qkv_w"][l].sum() == 3 * hd * dh * d
        assert G["proj_w"][l].sum() == d * hd * dh
        assert G["fc1_w"][l].sum() == dm * d and G["fc2_w"][l].sum() == d * dm


def test_update_keeps_the_previous_level_bit_identical(mini):
    w, x, t, y = mini
    for k in (0, 1):
        r = og.growth_step(w, MINI, t, k, x, y, lr=0.5, clip=1e9)
        before = oracle.elastic_forward(w, MINI, t, k + 1, x)
        after = oracle.elastic_forward(r["weights"], MINI, t, k + 1, x)
        np.testing.assert_array_equal(after, before)
        moved = oracle.elastic_forward(r["weights"], MINI, t, k, x)
        assert np.max(np.abs(moved - oracle.elastic_forward(w, MINI, t, k, x))) > 1e-6
        for key in w:                            # only masked entries move
            diff = r["weights"][key] != w[key]
            assert not (diff & (r["mask"][key] == 0)).any(), key


def test_clipping_bounds_the_step_and_is_selective(mini):
    w, x, t, y = mini
    free = og.growth_step(w, MINI, t, 0, x, y, lr=1.0, clip=1e9)
    assert free["scale"] == 1.0 and free["norm"] > 0
    c = 0.25 * free["norm"]
    cl = og.growth_step(w, MINI, t, 0, x, y, lr=1.0, clip=c)
    step = math.sqrt(sum(float(((cl["weights"][key] - w[key]) ** 2).sum()) for key in w))
    assert abs(step - c) <= 1e-9 * c
    assert abs(cl["scale"] - 0.25) < 1e-12
    # the norm is taken over G (.) grad only: the full gradient is larger
    _, grad = og.loss_and_grad(w, MINI, t, 0, x, y)
    full = math.sqrt(sum(float((a * a).sum()) for a in grad.values()))
    assert full > free["norm"] * 1.01


def test_small_step_lowers_the_mode_loss(mini):
    w, x, t, y = mini
    l0, _ = og.loss_and_grad(w, MINI, t, 1, x, y)
    r = og.growth_step(w, MINI, t, 1, x, y, lr=1e-3, clip=1e9)
    l1, _ = og.loss_and_grad(r["weights"], MINI, t, 1, x, y)
    assert l1 < l0
    # first order: the decrease is lr * |G (.) grad|^2
    assert abs((l0 - l1) - 1e-3 * r["norm"] ** 2) < 0.05 * 1e-3 * r["norm"] ** 2


def test_growth_rejects_the_core_and_embedding_changes():
    w = inputs.make_weights(CONFIGS["tiny_emb"])
    t = inputs.make_dn_table(CONFIGS["tiny_emb"])
    x = inputs.make_images(CONFIGS["tiny_emb"], 1)
    with pytest.raises(ValueError):
        og.growth_step(w, CONFIGS["tiny_emb"], t, 0, x, [0], 0.1, 1.0)   # embed 64 -> 48
    tm = mini_table()
    wm = inputs.make_weights(MINI)
    with pytest.raises(ValueError):
        og.growth_step(wm, MINI, tm, tm.num_modes - 1, inputs.make_images(MINI, 1), [0], 0.1, 1.0)


# ------------------------------------------------------------- mutants
def _ln_bwd_no_mean(dy, xhat, rstd, g):
    dxhat = dy * g
    n = xhat.shape[-1]
    dx = rstd * (dxhat - xhat * (dxhat * xhat).sum(axis=-1, keepdims=True) / n)
    axes = tuple(range(dy.ndim - 1))
    return dx, (dy * xhat).sum(axis=axes), dy.sum(axis=axes)


def _gelu_grad_phi_only(z):
    return 0.5 * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))


def _attn_bwd_no_rowsum(P, q, k, v, do, hd):
    dv = P.transpose(0, 1, 3, 2) @ do
    dS = P * (do @ v.transpose(0, 1, 3, 2)) / math.sqrt(hd)
    return dS @ k, dS.transpose(0, 1, 3, 2) @ q, dv


_ORIG_ATTN = og.attention_bwd


def _attn_bwd_dk_untransposed(P, q, k, v, do, hd):
    dq, _, dv = _ORIG_ATTN(P, q, k, v, do, hd)
    dP = do @ v.transpose(0, 1, 3, 2)
    dS = P * (dP - (dP * P).sum(axis=-1, keepdims=True)) / math.sqrt(hd)
    return dq, dS @ q, dv


@pytest.mark.parametrize("name,fn", [("layer_norm_bwd", _ln_bwd_no_mean),
                                     ("gelu_grad", _gelu_grad_phi_only),
                                     ("attention_bwd", _attn_bwd_no_rowsum),
                                     ("attention_bwd", _attn_bwd_dk_untransposed)],
                         ids=["ln-no-mean", "gelu-phi-only", "softmax-no-rowsum", "dk-untransposed"])
def test_autograd_pin_catches_planted_mistake(monkeypatch, mini, name, fn):
    monkeypatch.setattr(og, name, fn)
    with pytest.raises(AssertionError):
        test_gradient_matches_torch_autograd(mini, 0)
