"""Plain fp64 CPU oracle for the elastic-ViT forward pass.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run anything in this package.
It shares no code with the HIP path and imports nothing from it.

What it computes (Section 4.1 of the paper, which follows the original ViT):
an image is cut into (img/P)^2 non-overlapping P x P x C patches, each patch
is projected linearly to d, a class token is prepended and position
embeddings are added; L pre-norm encoder blocks follow, each one multi-head
self-attention (Eqs. 2-3) and a two-layer GELU MLP (Eq. 5) with residual
connections; the class token's final LayerNorm output goes through a linear
classifier.

A Descendant Network (DN) keeps a subset of heads and MLP hidden units per
layer.  Structured pruning masks whole rows/columns to zero (Eqs. 4 and 6);
nesting of the DNs (Eq. 8) makes each mode's active set a prefix of one
per-layer order.  Three formulations live here:

* ``vit_forward``            (F1) a dense ViT whose layers may have any number
                              of heads / MLP units;
* ``elastic_forward_masked`` (F2) the paper's literal form: full-width
                              weights multiplied by {0,1} masks, then F1;
* ``extract_dense``          (F3) copies the active sub-blocks into a smaller
                              dense ViT, which F1 then runs.

Readings where the paper is silent (each is listed in the design notes):
LayerNorm eps 1e-6 with biased variance; exact erf GELU; attention scale
1/sqrt(d/H) with H the full head count in every mode; a pruned head removes
its q/k/v output rows and its input columns of the output projection.  A
narrower embedding (Section 4.1 also reduces the hidden size of the
LayerNorm and patch-embedding layers) keeps one set of embedding channels in
every layer, and each LayerNorm normalises over that set only.

Parity status: pinned (see tests/test_oracle.py) by a textbook ViT built from
torch CPU fp64 library ops (full width), brute-force matmul / softmax /
LayerNorm checks, mask-form vs gather-form agreement, permutation invariance,
bias-mask irrelevance and locality.
"""
from __future__ import annotations

import math
from typing import Dict, List

import numpy as np
from scipy.special import erf

Params = Dict[str, object]


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis: mean, biased variance, affine."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def layer_norm_masked(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float,
                      m: np.ndarray) -> np.ndarray:
    """LayerNorm over the channels where the {0,1} mask m is 1 (mean and biased
    variance over those channels only); masked-out channels give 0."""
    n = m.sum()
    mu = (x * m).sum(axis=-1, keepdims=True) / n
    var = (((x - mu) * m) ** 2).sum(axis=-1, keepdims=True) / n
    return ((x - mu) / np.sqrt(var + eps) * g + b) * m


def gelu(z: np.ndarray) -> np.ndarray:
    """Exact GELU: z * Phi(z) with Phi the standard normal CDF (Eq. 5's phi)."""
    return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row-wise softmax over the last axis, max-subtracted (Eq. 3)."""
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def patchify(images: np.ndarray, patch: int) -> np.ndarray:
    """[B, C, H, W] -> [B, N, C*P*P]: patch n = row-major over the patch grid,
    features in (channel, row-in-patch, column-in-patch) order."""
    B, C, H, W = images.shape
    gh, gw = H // patch, W // patch
    x = images.reshape(B, C, gh, patch, gw, patch)
    x = x.transpose(0, 2, 4, 1, 3, 5)          # B, gy, gx, C, i, j
    return x.reshape(B, gh * gw, C * patch * patch)


def attention(u: np.ndarray, qkv_w: np.ndarray, qkv_b: np.ndarray,
              head_dim: int) -> np.ndarray:
    """Multi-head self-attention (Eqs. 2-3) up to, not including, W^O.

    qkv_w rows are [q heads | k heads | v heads], each head ``head_dim`` rows,
    so a layer with h heads has 3*h*head_dim rows.  Returns the concatenated
    head outputs [B, T, h*head_dim].
    """
    B, T, _ = u.shape
    h = qkv_w.shape[0] // (3 * head_dim)
    qkv = u @ qkv_w.T + qkv_b                   # [B, T, 3*h*hd]
    qkv = qkv.reshape(B, T, 3, h, head_dim).transpose(2, 0, 3, 1, 4)
    q, k, v = qkv[0], qkv[1], qkv[2]            # [B, h, T, hd]
    s = (q @ k.transpose(0, 1, 3, 2)) / math.sqrt(head_dim)
    p = softmax_rows(s)
    o = p @ v                                   # [B, h, T, hd]
    return o.transpose(0, 2, 1, 3).reshape(B, T, h * head_dim)


def vit_forward(p: Params, images: np.ndarray, head_dim: int, eps: float,
                embed_mask: np.ndarray = None) -> np.ndarray:
    """F1: dense ViT forward in fp64.  Returns logits [B, num_classes].

    ``p["layers"]`` is a list of per-layer dicts; each layer may have its own
    head count (rows of qkv_w / (3*head_dim)) and MLP width (rows of fc1_w).
    With ``embed_mask`` (a {0,1} vector over the d channels) every LayerNorm
    normalises over the unmasked channels only (F2's form of a narrower
    embedding); the masked weights themselves are the caller's.
    """
    f = lambda a: np.asarray(a, dtype=np.float64)
    if embed_mask is None:
        ln = layer_norm
    else:
        ln = lambda x, g, b, e: layer_norm_masked(x, g, b, e, embed_mask)
    x = patchify(f(images), int(f(p["patch_w"]).shape[-1]))
    d = f(p["patch_w"]).shape[0]
    e = x @ f(p["patch_w"]).reshape(d, -1).T + f(p["patch_b"])
    B = e.shape[0]
    cls = np.broadcast_to(f(p["cls"]), (B, 1, d))
    x = np.concatenate([cls, e], axis=1) + f(p["pos"])
    for lp in p["layers"]:
        u = ln(x, f(lp["ln1_g"]), f(lp["ln1_b"]), eps)
        o = attention(u, f(lp["qkv_w"]), f(lp["qkv_b"]), head_dim)
        x = x + (o @ f(lp["proj_w"]).T + f(lp["proj_b"]))
        u = ln(x, f(lp["ln2_g"]), f(lp["ln2_b"]), eps)
        g = gelu(u @ f(lp["fc1_w"]).T + f(lp["fc1_b"]))
        x = x + (g @ f(lp["fc2_w"]).T + f(lp["fc2_b"]))
    c = ln(x[:, 0], f(p["norm_g"]), f(p["norm_b"]), eps)
    return c @ f(p["head_w"]).T + f(p["head_b"])


def canonical_params(w: Dict[str, np.ndarray], depth: int) -> Params:
    """Stacked canonical arrays (layer on axis 0) -> F1's nested form, fp64."""
    f = lambda a: np.asarray(a, dtype=np.float64)
    keys = ("ln1_g", "ln1_b", "qkv_w", "qkv_b", "proj_w", "proj_b",
            "ln2_g", "ln2_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")
    p: Params = {k: f(w[k]) for k in ("patch_w", "patch_b", "cls", "pos",
                                      "norm_g", "norm_b", "head_w", "head_b")}
    p["layers"] = [{k: f(w[k][l]) for k in keys} for l in range(depth)]
    return p


def active_sets(table, k: int, layer: int):
    """Active head and MLP-unit indices of mode k in one layer, in order."""
    h = int(table.n_heads[k][layer])
    m = int(table.n_mlp[k][layer])
    return (np.asarray(table.head_order[layer][:h], dtype=np.int64),
            np.asarray(table.mlp_order[layer][:m], dtype=np.int64))


def active_embed(table, k: int, dim: int) -> np.ndarray:
    """Active embedding channels of mode k, in order (all d when the table
    narrows no embedding)."""
    order = getattr(table, "embed_order", None)
    n_embed = getattr(table, "n_embed", None)
    order = np.arange(dim) if order is None else np.asarray(order, dtype=np.int64)
    n = dim if n_embed is None else int(n_embed[k])
    return order[:n]


def embed_mask(table, k: int, dim: int) -> np.ndarray:
    """{0,1} mask over the d embedding channels of mode k."""
    m = np.zeros(dim)
    m[active_embed(table, k, dim)] = 1.0
    return m


def masks(table, k: int, layer: int, dim: int, heads: int, mlp_hidden: int):
    """Binary masks of Eqs. 4 and 6 for one layer of mode k.

    Returns (m_qkv_rows [3d], m_proj_cols [d], m_fc1_rows [M], m_fc2_cols [M]):
    a pruned head zeroes its q/k/v rows and its proj input columns; a pruned
    MLP unit zeroes its fc1 row and its fc2 column.
    """
    hd = dim // heads
    act_h, act_m = active_sets(table, k, layer)
    head_on = np.zeros(heads)
    head_on[act_h] = 1.0
    unit_on = np.zeros(mlp_hidden)
    unit_on[act_m] = 1.0
    per_chan = np.repeat(head_on, hd)            # [d]: channel c belongs to head c // hd
    return np.tile(per_chan, 3), per_chan, unit_on, unit_on


def elastic_forward_masked(w: Dict[str, np.ndarray], cfg, table, k: int,
                           images: np.ndarray, mask_biases: bool = True) -> np.ndarray:
    """F2: mode-k logits as M (.) W on the full-width model, then F1 (Eqs. 4, 6).

    A narrower embedding masks every embedding channel outside the active set:
    patch-embedding rows, class token, positions, the input columns of q/k/v
    and fc1, the output rows of the projection and fc2 (with their biases),
    the classifier's input columns, and the LayerNorm affine parameters; every
    LayerNorm then normalises over the active channels only.  Masked channels
    of the residual stream stay exactly zero.
    """
    p = canonical_params(w, cfg.depth)
    me = embed_mask(table, k, cfg.dim)
    narrow = me.sum() < cfg.dim
    if narrow:
        p["patch_w"] = p["patch_w"] * me[:, None, None, None]
        p["patch_b"] = p["patch_b"] * me
        p["cls"] = p["cls"] * me
        p["pos"] = p["pos"] * me[None, :]
        p["norm_g"] = p["norm_g"] * me
        p["norm_b"] = p["norm_b"] * me
        p["head_w"] = p["head_w"] * me[None, :]
    for l, lp in enumerate(p["layers"]):
        mq, mo, m1, m2 = masks(table, k, l, cfg.dim, cfg.heads, cfg.mlp_hidden)
        lp["qkv_w"] = mq[:, None] * lp["qkv_w"]
        lp["proj_w"] = lp["proj_w"] * mo[None, :]
        lp["fc1_w"] = m1[:, None] * lp["fc1_w"]
        lp["fc2_w"] = lp["fc2_w"] * m2[None, :]
        if mask_biases:
            lp["qkv_b"] = mq * lp["qkv_b"]
            lp["fc1_b"] = m1 * lp["fc1_b"]
        if narrow:
            lp["qkv_w"] = lp["qkv_w"] * me[None, :]
            lp["fc1_w"] = lp["fc1_w"] * me[None, :]
            lp["proj_w"] = me[:, None] * lp["proj_w"]
            lp["proj_b"] = me * lp["proj_b"]
            lp["fc2_w"] = me[:, None] * lp["fc2_w"]
            lp["fc2_b"] = me * lp["fc2_b"]
            for key in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
                lp[key] = me * lp[key]
    return vit_forward(p, images, cfg.dim // cfg.heads, cfg.ln_eps,
                       embed_mask=me if narrow else None)


def extract_dense(w: Dict[str, np.ndarray], cfg, table, k: int) -> Params:
    """F3: copy mode k's active sub-blocks, in order, into a smaller dense ViT."""
    p = canonical_params(w, cfg.depth)
    d, hd = cfg.dim, cfg.dim // cfg.heads
    e = active_embed(table, k, d)
    p["patch_w"] = p["patch_w"][e].copy()
    p["patch_b"] = p["patch_b"][e].copy()
    p["cls"] = p["cls"][e].copy()
    p["pos"] = p["pos"][:, e].copy()
    p["norm_g"] = p["norm_g"][e].copy()
    p["norm_b"] = p["norm_b"][e].copy()
    p["head_w"] = p["head_w"][:, e].copy()
    for l, lp in enumerate(p["layers"]):
        act_h, act_m = active_sets(table, k, l)
        chans = np.concatenate([np.arange(i * hd, (i + 1) * hd) for i in act_h])
        rows = np.concatenate([chans, d + chans, 2 * d + chans])
        lp["qkv_w"] = lp["qkv_w"][rows][:, e].copy()
        lp["qkv_b"] = lp["qkv_b"][rows].copy()
        lp["proj_w"] = lp["proj_w"][e][:, chans].copy()
        lp["proj_b"] = lp["proj_b"][e].copy()
        lp["fc1_w"] = lp["fc1_w"][act_m][:, e].copy()
        lp["fc1_b"] = lp["fc1_b"][act_m].copy()
        lp["fc2_w"] = lp["fc2_w"][e][:, act_m].copy()
        lp["fc2_b"] = lp["fc2_b"][e].copy()
        for key in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
            lp[key] = lp[key][e].copy()
    return p


def elastic_forward(w: Dict[str, np.ndarray], cfg, table, k: int,
                    images: np.ndarray, chunk: int = 16) -> np.ndarray:
    """Mode-k logits via F3 + F1, in image chunks (the fast form used for expected values)."""
    p = extract_dense(w, cfg, table, k)
    hd = cfg.dim // cfg.heads
    outs: List[np.ndarray] = []
    for s in range(0, images.shape[0], chunk):
        outs.append(vit_forward(p, images[s:s + chunk], hd, cfg.ln_eps))
    return np.concatenate(outs, axis=0)
