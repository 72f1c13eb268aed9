"""Planted mistakes in the oracle (on the CPU) must be caught by its pins.

Each mutant replaces one oracle function with a plausible wrong version (a
dropped term, a wrong scale, a transposed operand, a wrong index); the pin
that guards it must then fail.  This shows the pins are not vacuous.
"""
import math

import numpy as np
import pytest

import oracle
import oracle.vit as ov
from paper_2609_10018_amd import inputs
from paper_2609_10018_amd.inputs import CONFIGS
from test_oracle import MINI, mini_table
from textbook import loop_extract_embed, loop_masked_weights, rel_err, torch_vit

_orig = {name: getattr(ov, name) for name in
         ("layer_norm", "gelu", "softmax_rows", "patchify", "attention", "active_sets",
          "masks", "layer_norm_masked", "active_embed")}


def _ln_no_beta(x, g, b, eps):
    return _orig["layer_norm"](x, g, np.zeros_like(b), eps)


def _ln_unbiased(x, g, b, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)
    return (x - mu) / np.sqrt(var + eps) * g + b


def _gelu_tanh(z):
    return 0.5 * z * (1 + np.tanh(math.sqrt(2 / math.pi) * (z + 0.044715 * z ** 3)))


def _patchify_ji(images, patch):
    B, C, H, W = images.shape
    g = H // patch
    x = images.reshape(B, C, g, patch, g, patch).transpose(0, 2, 4, 1, 5, 3)
    return x.reshape(B, g * g, C * patch * patch)


def _attention_scale_hd(u, qkv_w, qkv_b, head_dim):
    return _attn_with_scale(u, qkv_w, qkv_b, head_dim, 1.0 / head_dim)


def _attn_with_scale(u, qkv_w, qkv_b, head_dim, scale, swap_qk=False, interleaved=False):
    B, T, _ = u.shape
    h = qkv_w.shape[0] // (3 * head_dim)
    qkv = u @ qkv_w.T + qkv_b
    if interleaved:
        qkv = qkv.reshape(B, T, h, 3, head_dim).transpose(3, 0, 2, 1, 4)
    else:
        qkv = qkv.reshape(B, T, 3, h, head_dim).transpose(2, 0, 3, 1, 4)
    q, k, v = qkv[0], qkv[1], qkv[2]
    if swap_qk:
        s = (k @ q.transpose(0, 1, 3, 2)) * scale
    else:
        s = (q @ k.transpose(0, 1, 3, 2)) * scale
    p = ov.softmax_rows(s)
    return (p @ v).transpose(0, 2, 1, 3).reshape(B, T, h * head_dim)


def _attention_swapped_qk(u, qkv_w, qkv_b, head_dim):
    return _attn_with_scale(u, qkv_w, qkv_b, head_dim, 1 / math.sqrt(head_dim), swap_qk=True)


def _attention_interleaved(u, qkv_w, qkv_b, head_dim):
    return _attn_with_scale(u, qkv_w, qkv_b, head_dim, 1 / math.sqrt(head_dim), interleaved=True)


def _softmax_cols(s):
    e = np.exp(s - s.max(axis=-2, keepdims=True))
    return e / e.sum(axis=-2, keepdims=True)


def _active_suffix(table, k, layer):
    h = int(table.n_heads[k][layer])
    m = int(table.n_mlp[k][layer])
    H = len(table.head_order[layer])
    M = len(table.mlp_order[layer])
    return (np.asarray(table.head_order[layer][H - h:], dtype=np.int64),
            np.asarray(table.mlp_order[layer][M - m:], dtype=np.int64))


def _masks_modulo(table, k, layer, dim, heads, mlp_hidden):
    hd = dim // heads
    act_h, act_m = _orig["active_sets"](table, k, layer)
    on = np.zeros(heads)
    on[act_h] = 1.0
    per_chan = on[np.arange(dim) % heads]         # wrong channel -> head map
    unit_on = np.zeros(mlp_hidden)
    unit_on[act_m] = 1.0
    return np.tile(per_chan, 3), per_chan, unit_on, unit_on


def _full_width_err(cfg):
    w = inputs.make_weights(cfg)
    x = inputs.make_images(cfg, 2)
    got = oracle.vit_forward(oracle.canonical_params(w, cfg.depth), x,
                             cfg.dim // cfg.heads, cfg.ln_eps)
    return rel_err(got, torch_vit(w, x, cfg))


def _masked_mode_err():
    w = inputs.make_weights(MINI)
    x = inputs.make_images(MINI, 2)
    table = mini_table()
    errs = []
    for k in range(1, table.num_modes):
        ref = torch_vit(loop_masked_weights(w, MINI, table, k), x, MINI)
        errs.append(rel_err(oracle.elastic_forward(w, MINI, table, k, x), ref))
    return max(errs)


def _c2_err():
    w = inputs.make_weights(MINI)
    x = inputs.make_images(MINI, 2)
    table = mini_table()
    return max(rel_err(oracle.elastic_forward(w, MINI, table, k, x),
                       oracle.elastic_forward_masked(w, MINI, table, k, x))
               for k in range(1, table.num_modes))


def _ln_masked_full_stats(x, g, b, eps, m):
    return _orig["layer_norm"](x, g, b, eps) * m      # statistics over all d channels


def _active_embed_suffix(table, k, dim):
    order = np.asarray(table.embed_order, dtype=np.int64)
    return order[dim - int(table.n_embed[k]):]


def _embed_err(form):
    import dataclasses
    cfg = CONFIGS["tiny_emb"]
    w = inputs.make_weights(cfg)
    x = inputs.make_images(cfg, 2)
    table = inputs.make_dn_table(cfg)
    errs = []
    for k in range(1, table.num_modes):
        sub, E = loop_extract_embed(w, cfg, table, k)
        ref = torch_vit(sub, x, dataclasses.replace(cfg, dim=E), head_dim=cfg.head_dim)
        errs.append(rel_err(form(w, cfg, table, k, x), ref))
    return max(errs)


def _embed_mask_form_err():
    return _embed_err(oracle.elastic_forward_masked)


def _embed_gather_form_err():
    return _embed_err(oracle.elastic_forward)


MUTANTS = [
    ("layer_norm", _ln_no_beta, _full_width_err),
    ("layer_norm", _ln_unbiased, _full_width_err),
    ("gelu", _gelu_tanh, _full_width_err),
    ("patchify", _patchify_ji, _full_width_err),
    ("attention", _attention_scale_hd, _full_width_err),
    ("attention", _attention_swapped_qk, _full_width_err),
    ("attention", _attention_interleaved, _full_width_err),
    ("softmax_rows", _softmax_cols, _full_width_err),
    ("active_sets", _active_suffix, _masked_mode_err),
    ("masks", _masks_modulo, _c2_err),
    ("layer_norm_masked", _ln_masked_full_stats, _embed_mask_form_err),
    ("active_embed", _active_embed_suffix, _embed_gather_form_err),
]


@pytest.mark.parametrize("name,mutant,check", MUTANTS,
                         ids=[f"{n}-{m.__name__}" for n, m, _ in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, mutant, check):
    assert check(MINI) < 1e-10 if check is _full_width_err else check() < 1e-10
    monkeypatch.setattr(ov, name, mutant)
    err = check(MINI) if check is _full_width_err else check()
    assert err > 1e-6, f"mutant {mutant.__name__} of {name} went undetected (err {err})"
