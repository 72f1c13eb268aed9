"""Algorithmic work of one elastic-ViT forward per image, per DN mode.

FLOPs are 2 x multiply-accumulates of the dense contractions: patch embedding,
q/k/v, attention QK^T and PV, output projection, fc1, fc2 and the classifier,
every token counted in every layer.  Element-wise work (LayerNorm, GELU,
softmax, adds) is not counted.  ``paper_macs`` is the convention that matches
the base ViT-B figure of Table 1: linear-layer MACs only (no QK^T / PV).

``layernorm_bytes_per_image`` is the algorithmic HBM traffic of a standalone
LayerNorm over every token (read one residual-stream row, write one LayerNorm
output row): the fp32 path runs one per block input; the bf16 path folds the
per-block LayerNorms into the next GEMM and runs only the final one, on the
class-token rows.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from .inputs import ModelConfig


def layer_widths(table, k: int):
    return (np.asarray(table.n_heads[k], dtype=np.int64),
            np.asarray(table.n_mlp[k], dtype=np.int64))


def embed_width(cfg: ModelConfig, table, k: int) -> int:
    """Active embedding channels of mode k (all d when the table has none)."""
    n = getattr(table, "n_embed", None)
    return cfg.dim if n is None else int(n[k])


def gemm_flops(cfg: ModelConfig, table, k: int) -> Dict[str, float]:
    """Per-image FLOPs of each contraction kernel class in mode k."""
    T, d, hd = cfg.tokens, embed_width(cfg, table, k), cfg.head_dim
    h, m = layer_widths(table, k)
    return {
        "patch": 2.0 * cfg.num_patches * cfg.patch_k * d,
        "qkv": float(np.sum(2.0 * T * d * 3 * hd * h)),
        "attn": float(np.sum(2.0 * 2 * T * T * hd * h)),
        "proj": float(np.sum(2.0 * T * hd * h * d)),
        "fc1": float(np.sum(2.0 * T * d * m)),
        "fc2": float(np.sum(2.0 * T * m * d)),
        "head": 2.0 * d * cfg.num_classes,
    }


def flops_per_image(cfg: ModelConfig, table, k: int) -> float:
    return float(sum(gemm_flops(cfg, table, k).values()))


def growth_step_flops(cfg: ModelConfig, table, k: int) -> float:
    """Per-image FLOPs of one growth step of mode k from mode k + 1 (Eq. 9)
    as the bf16 path runs it: the mode-k forward (gemm_flops); the
    activation-gradient contractions of the head and of every layer's fc2,
    fc1, projection and q/k/v over mode k's widths; the attention backward
    counted as five T x T x head_dim contractions per head (the scores once
    recomputed, dP, dV, dQ, dK); and the weight-gradient contractions over
    the re-introduced slices only (mode k's widths minus mode k + 1's).  The
    patch embedding is not differentiated."""
    T, d, hd = cfg.tokens, embed_width(cfg, table, k), cfg.head_dim
    h, m = layer_widths(table, k)
    hp, mp = layer_widths(table, k + 1)
    act = 2.0 * T * (d * m + m * d + d * hd * h + 3 * hd * h * d)
    attn = 5 * 2.0 * T * T * hd * h
    wgrad = 2.0 * T * (d * (m - mp) + (m - mp) * d + d * hd * (h - hp) + 3 * hd * (h - hp) * d)
    return (flops_per_image(cfg, table, k) + 2.0 * d * cfg.num_classes
            + float(np.sum(act + attn + wgrad)))


def paper_macs(cfg: ModelConfig, table, k: int) -> float:
    f = gemm_flops(cfg, table, k)
    return (f["patch"] + f["qkv"] + f["proj"] + f["fc1"] + f["fc2"] + f["head"]) / 2.0


def layernorm_bytes_per_image(cfg: ModelConfig, in_bytes: int = 4, out_bytes: int = 4) -> float:
    """One standalone LayerNorm over all tokens: read T*d inputs + write T*d
    outputs (element sizes in bytes; fp32 path: 4 and 4)."""
    return cfg.tokens * cfg.dim * float(in_bytes + out_bytes)


def active_weight_elems(cfg: ModelConfig, table, k: int) -> int:
    """Matrix elements a mode-k forward reads (biases and norms excluded)."""
    d, hd, C = embed_width(cfg, table, k), cfg.head_dim, cfg.num_classes
    h, m = layer_widths(table, k)
    per_layer = 3 * hd * h * d + d * hd * h + m * d + d * m
    return int(d * cfg.patch_k + per_layer.sum() + C * d)


def dense_model_bytes(cfg: ModelConfig, table, k: int, matrix_bytes: int = 2,
                      vector_bytes: int = 4) -> int:
    """Bytes of mode k as a dense model of its own (the DN's weights copied
    out, as a bag of per-mode models would store it): matrices at
    matrix_bytes per element, biases, norms, class token and positions at
    vector_bytes."""
    d, hd, C, T = embed_width(cfg, table, k), cfg.head_dim, cfg.num_classes, cfg.tokens
    h, m = layer_widths(table, k)
    vec = 2 * d + T * d + 2 * d + C                          # patch_b, cls, pos, norm, head_b
    vec += int(np.sum(2 * d + 3 * hd * h + d + 2 * d + m + d))  # per layer: ln1, bqkv, bo, ln2, b1, b2
    return int(active_weight_elems(cfg, table, k) * matrix_bytes + vec * vector_bytes)


def cnn_layer_macs(cfg, table, k: int):
    """Per-image MACs of each convolution of an elastic bottleneck ResNet in
    mode k, in forward order: (name, MACs)."""
    out = []
    hw = cfg.img // 2
    out.append(("stem", hw * hw * cfg.stem * cfg.in_chans * 49))
    hw //= 2
    for i, b in enumerate(cfg.block_specs()):
        w = int(table.n_width[k][i])
        ho = hw // b["stride"]
        out.append((f"b{i}_c1", hw * hw * w * b["c_in"]))
        out.append((f"b{i}_c2", ho * ho * w * w * 9))
        out.append((f"b{i}_c3", ho * ho * b["c_out"] * w))
        if b["down"]:
            out.append((f"b{i}_dn", ho * ho * b["c_out"] * b["c_in"]))
        hw = ho
    out.append(("fc", cfg.features * cfg.num_classes))
    return out


def cnn_macs(cfg, table, k: int) -> int:
    """Per-image multiply-accumulates of every convolution and the classifier."""
    return int(sum(m for _, m in cnn_layer_macs(cfg, table, k)))
