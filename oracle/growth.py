"""Plain fp64 CPU oracle of one growth step of the elastic ViT.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run anything in this package.
It shares no code with the HIP path and imports nothing from it.

What it computes (Section 4.2, Eqs. 8 and 9 and the selective gradient
clipping that follows them).  Growing the DN of mode k re-introduces the
weights that mode k has and the next smaller mode k+1 (the previous level)
lacks; the weights of mode k+1 are shared and stay frozen.  One step:

1. the mode-k forward (the DN as a dense network, F3 + F1 of ``vit``) and the
   mean cross-entropy of its logits against integer labels;
2. the gradient of that loss with respect to every weight of the DN, by the
   chain rule written out layer by layer (``backward``);
3. Eq. 9's mask G: 1 on the re-introduced weights (q/k/v rows and biases of
   the heads active in mode k but not in k+1, those heads' input columns of
   the output projection; fc1 rows and biases and fc2 columns of the MLP
   units active in k but not in k+1), 0 on every weight that mode k+1 holds;
4. selective clipping: G (.) grad is rescaled to L2 norm at most ``clip``
   (norm clipping, the method the paper cites), only these entries take part;
5. W <- W - lr * (clipped G (.) grad).

Weights outside mode k are not part of the DN and are left as they are.
Growth keeps every mode's embedding width (the embedding is not grown here):
``growth_step`` rejects tables whose modes k and k+1 differ in it.

Parity status: pinned in tests/test_oracle_growth.py by central finite
differences of the loss, by torch CPU fp64 autograd through the textbook ViT,
by the invariance of mode k+1's logits under the update, by the count and
placement of the mask's ones and by the clipping bound; planted mistakes in
the backward fail those pins.
"""
from __future__ import annotations

import math
from typing import Dict, List, Tuple

import numpy as np
from scipy.special import erf

from . import vit as _vit

LAYER_KEYS = ("ln1_g", "ln1_b", "qkv_w", "qkv_b", "proj_w", "proj_b",
              "ln2_g", "ln2_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")
GLOBAL_KEYS = ("patch_w", "patch_b", "cls", "pos", "norm_g", "norm_b", "head_w", "head_b")


# ----------------------------------------------------------------- pieces
def layer_norm_fwd(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float):
    """LayerNorm over the last axis (biased variance); returns (y, xhat, rstd)."""
    mu = x.mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(((x - mu) ** 2).mean(axis=-1, keepdims=True) + eps)
    xhat = (x - mu) * rstd
    return xhat * g + b, xhat, rstd


def layer_norm_bwd(dy: np.ndarray, xhat: np.ndarray, rstd: np.ndarray, g: np.ndarray):
    """Gradients of y = xhat * g + b: (dx, dg, db), dg / db summed over rows."""
    dxhat = dy * g
    n = xhat.shape[-1]
    dx = rstd * (dxhat - dxhat.sum(axis=-1, keepdims=True) / n
                 - xhat * (dxhat * xhat).sum(axis=-1, keepdims=True) / n)
    axes = tuple(range(dy.ndim - 1))
    return dx, (dy * xhat).sum(axis=axes), dy.sum(axis=axes)


def gelu(z: np.ndarray) -> np.ndarray:
    return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))


def gelu_grad(z: np.ndarray) -> np.ndarray:
    """d/dz of z * Phi(z): Phi(z) + z * phi(z)."""
    return 0.5 * (1.0 + erf(z / math.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / math.sqrt(2 * math.pi)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def cross_entropy(logits: np.ndarray, labels: np.ndarray):
    """Mean over the batch of -log softmax(logits)[label]; returns (loss, dlogits)."""
    B = logits.shape[0]
    z = logits - logits.max(axis=1, keepdims=True)
    logp = z - np.log(np.exp(z).sum(axis=1, keepdims=True))
    loss = -logp[np.arange(B), labels].mean()
    d = np.exp(logp)
    d[np.arange(B), labels] -= 1.0
    return float(loss), d / B


def attention_bwd(P, q, k, v, do, head_dim: int):
    """Gradients of o = softmax(q k^T / sqrt(hd)) v per (image, head):
    dv = P^T do; dS = P (.) (dP - rowsum(dP (.) P)) / sqrt(hd) with dP = do v^T
    (softmax's Jacobian); dq = dS k, dk = dS^T q."""
    dv = P.transpose(0, 1, 3, 2) @ do
    dP = do @ v.transpose(0, 1, 3, 2)
    dS = P * (dP - (dP * P).sum(axis=-1, keepdims=True)) / math.sqrt(head_dim)
    return dS @ k, dS.transpose(0, 1, 3, 2) @ q, dv


# --------------------------------------------------------- forward / backward
def forward(p: dict, images: np.ndarray, head_dim: int, eps: float):
    """F1 forward of a dense ViT (``vit.canonical_params`` form) that keeps what
    the backward needs.  Returns (logits, cache)."""
    f = lambda a: np.asarray(a, dtype=np.float64)
    patches = _vit.patchify(f(images), int(f(p["patch_w"]).shape[-1]))
    d = f(p["patch_w"]).shape[0]
    B = patches.shape[0]
    e = patches @ f(p["patch_w"]).reshape(d, -1).T + f(p["patch_b"])
    x = np.concatenate([np.broadcast_to(f(p["cls"]), (B, 1, d)), e], axis=1) + f(p["pos"])
    cache = {"patches": patches, "layers": []}
    for lp in p["layers"]:
        c: dict = {"x_in": x}
        u1, c["xhat1"], c["rstd1"] = layer_norm_fwd(x, lp["ln1_g"], lp["ln1_b"], eps)
        c["u1"] = u1
        h = lp["qkv_w"].shape[0] // (3 * head_dim)
        T = x.shape[1]
        qkv = (u1 @ lp["qkv_w"].T + lp["qkv_b"]).reshape(B, T, 3, h, head_dim)
        q, k, v = (qkv[:, :, i].transpose(0, 2, 1, 3) for i in range(3))   # [B, h, T, hd]
        P = softmax_rows(q @ k.transpose(0, 1, 3, 2) / math.sqrt(head_dim))
        o = (P @ v).transpose(0, 2, 1, 3).reshape(B, T, h * head_dim)
        c.update(q=q, k=k, v=v, P=P, o=o, h=h)
        x = x + o @ lp["proj_w"].T + lp["proj_b"]
        c["x_mid"] = x
        u2, c["xhat2"], c["rstd2"] = layer_norm_fwd(x, lp["ln2_g"], lp["ln2_b"], eps)
        c["u2"] = u2
        z = u2 @ lp["fc1_w"].T + lp["fc1_b"]
        g = gelu(z)
        c.update(z=z, g=g)
        x = x + g @ lp["fc2_w"].T + lp["fc2_b"]
        cache["layers"].append(c)
    cache["x_out"] = x
    cn, cache["xhatf"], cache["rstdf"] = layer_norm_fwd(x[:, 0], p["norm_g"], p["norm_b"], eps)
    cache["cn"] = cn
    return cn @ p["head_w"].T + p["head_b"], cache


def backward(p: dict, cache: dict, dlogits: np.ndarray, head_dim: int) -> dict:
    """Gradient of a scalar loss with dL/dlogits = ``dlogits`` with respect to
    every weight of the dense ViT ``p``, in the same nested form."""
    grads: dict = {"layers": [None] * len(p["layers"])}
    grads["head_w"] = dlogits.T @ cache["cn"]
    grads["head_b"] = dlogits.sum(axis=0)
    dcn = dlogits @ p["head_w"]
    dx0, grads["norm_g"], grads["norm_b"] = layer_norm_bwd(dcn, cache["xhatf"], cache["rstdf"],
                                                           p["norm_g"])
    dx = np.zeros_like(cache["x_out"])
    dx[:, 0] = dx0
    rows = lambda a: a.reshape(-1, a.shape[-1])      # [B, T, n] -> [B*T, n]
    for l in range(len(p["layers"]) - 1, -1, -1):
        lp, c = p["layers"][l], cache["layers"][l]
        gl: dict = {}
        # MLP: x_out = x_mid + gelu(u2 W1^T + b1) W2^T + b2
        gl["fc2_w"] = rows(dx).T @ rows(c["g"])
        gl["fc2_b"] = rows(dx).sum(axis=0)
        dz = (dx @ lp["fc2_w"]) * gelu_grad(c["z"])
        gl["fc1_w"] = rows(dz).T @ rows(c["u2"])
        gl["fc1_b"] = rows(dz).sum(axis=0)
        du2 = dz @ lp["fc1_w"]
        dln, gl["ln2_g"], gl["ln2_b"] = layer_norm_bwd(du2, c["xhat2"], c["rstd2"], lp["ln2_g"])
        dx = dx + dln
        # attention: x_mid = x_in + o Wp^T + bp
        gl["proj_w"] = rows(dx).T @ rows(c["o"])
        gl["proj_b"] = rows(dx).sum(axis=0)
        B, T, _ = dx.shape
        h = c["h"]
        do = (dx @ lp["proj_w"]).reshape(B, T, h, head_dim).transpose(0, 2, 1, 3)
        dq, dk, dv = attention_bwd(c["P"], c["q"], c["k"], c["v"], do, head_dim)
        dqkv = np.stack([t.transpose(0, 2, 1, 3) for t in (dq, dk, dv)], axis=2)
        dqkv = dqkv.reshape(B, T, 3 * h * head_dim)
        gl["qkv_w"] = rows(dqkv).T @ rows(c["u1"])
        gl["qkv_b"] = rows(dqkv).sum(axis=0)
        du1 = dqkv @ lp["qkv_w"]
        dln, gl["ln1_g"], gl["ln1_b"] = layer_norm_bwd(du1, c["xhat1"], c["rstd1"], lp["ln1_g"])
        dx = dx + dln
        grads["layers"][l] = gl
    # embedding: x0 = [cls; patches Wpe^T + bpe] + pos
    grads["pos"] = dx.sum(axis=0)
    grads["cls"] = dx[:, 0].sum(axis=0)
    de = dx[:, 1:]
    d = p["patch_w"].shape[0]
    grads["patch_w"] = (rows(de).T @ rows(cache["patches"])).reshape(p["patch_w"].shape)
    grads["patch_b"] = rows(de).sum(axis=0)
    return grads


# ------------------------------------------------------ mapping and masks
def _chans(heads, hd):
    return np.concatenate([np.arange(i * hd, (i + 1) * hd) for i in heads]) if len(heads) else \
        np.zeros(0, dtype=np.int64)


def dense_to_canonical(grads: dict, cfg, table, k: int) -> Dict[str, np.ndarray]:
    """Scatter the gradient of mode k's dense DN (F3 order) into canonical
    full-width arrays (zeros where mode k has no weight)."""
    d, hd = cfg.dim, cfg.dim // cfg.heads
    e = _vit.active_embed(table, k, d)
    out: Dict[str, np.ndarray] = {}
    shapes = {"patch_w": (d, cfg.in_chans, cfg.patch, cfg.patch), "patch_b": (d,), "cls": (d,),
              "pos": (cfg.tokens, d), "norm_g": (d,), "norm_b": (d,),
              "head_w": (cfg.num_classes, d), "head_b": (cfg.num_classes,)}
    for key, shp in shapes.items():
        out[key] = np.zeros(shp)
    out["patch_w"][e] = grads["patch_w"]
    out["patch_b"][e] = grads["patch_b"]
    out["cls"][e] = grads["cls"]
    out["pos"][:, e] = grads["pos"]
    out["norm_g"][e] = grads["norm_g"]
    out["norm_b"][e] = grads["norm_b"]
    out["head_w"][:, e] = grads["head_w"]
    out["head_b"][:] = grads["head_b"]
    L, M = cfg.depth, cfg.mlp_hidden
    lshape = {"ln1_g": (d,), "ln1_b": (d,), "qkv_w": (3 * d, d), "qkv_b": (3 * d,),
              "proj_w": (d, d), "proj_b": (d,), "ln2_g": (d,), "ln2_b": (d,),
              "fc1_w": (M, d), "fc1_b": (M,), "fc2_w": (d, M), "fc2_b": (d,)}
    for key, shp in lshape.items():
        out[key] = np.zeros((L,) + shp)
    for l in range(L):
        act_h, act_m = _vit.active_sets(table, k, l)
        ch = _chans(act_h, hd)
        qrows = np.concatenate([ch, d + ch, 2 * d + ch])
        gl = grads["layers"][l]
        for key in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "proj_b", "fc2_b"):
            out[key][l][e] = gl[key]
        out["qkv_w"][l][np.ix_(qrows, e)] = gl["qkv_w"]
        out["qkv_b"][l][qrows] = gl["qkv_b"]
        out["proj_w"][l][np.ix_(e, ch)] = gl["proj_w"]
        out["fc1_w"][l][np.ix_(act_m, e)] = gl["fc1_w"]
        out["fc1_b"][l][act_m] = gl["fc1_b"]
        out["fc2_w"][l][np.ix_(e, act_m)] = gl["fc2_w"]
    return out


def growth_mask(cfg, table, k: int) -> Dict[str, np.ndarray]:
    """Eq. 9's G for growing mode k from mode k+1, in canonical shapes: 1 on
    the weights mode k re-introduces, 0 elsewhere."""
    d, hd, L, M = cfg.dim, cfg.dim // cfg.heads, cfg.depth, cfg.mlp_hidden
    G = {key: np.zeros(shp) for key, shp in _canonical_shapes(cfg).items()}
    e = _vit.active_embed(table, k, d)
    for l in range(L):
        heads_k, units_k = _vit.active_sets(table, k, l)
        heads_p, units_p = _vit.active_sets(table, k + 1, l)
        new_h = np.setdiff1d(heads_k, heads_p)
        new_m = np.setdiff1d(units_k, units_p)
        ch = _chans(new_h, hd)
        qrows = np.concatenate([ch, d + ch, 2 * d + ch])
        G["qkv_w"][l][np.ix_(qrows, e)] = 1.0
        G["qkv_b"][l][qrows] = 1.0
        G["proj_w"][l][np.ix_(e, ch)] = 1.0
        G["fc1_w"][l][np.ix_(new_m, e)] = 1.0
        G["fc1_b"][l][new_m] = 1.0
        G["fc2_w"][l][np.ix_(e, new_m)] = 1.0
    return G


def _canonical_shapes(cfg) -> Dict[str, tuple]:
    d, L, M, C = cfg.dim, cfg.depth, cfg.mlp_hidden, cfg.num_classes
    s = {"patch_w": (d, cfg.in_chans, cfg.patch, cfg.patch), "patch_b": (d,), "cls": (d,),
         "pos": (cfg.tokens, d), "norm_g": (d,), "norm_b": (d,), "head_w": (C, d), "head_b": (C,)}
    layer = {"ln1_g": (d,), "ln1_b": (d,), "qkv_w": (3 * d, d), "qkv_b": (3 * d,),
             "proj_w": (d, d), "proj_b": (d,), "ln2_g": (d,), "ln2_b": (d,),
             "fc1_w": (M, d), "fc1_b": (M,), "fc2_w": (d, M), "fc2_b": (d,)}
    s.update({key: (L,) + shp for key, shp in layer.items()})
    return s


# ------------------------------------------------------------- one step
def loss_and_grad(w: Dict[str, np.ndarray], cfg, table, k: int, images: np.ndarray,
                  labels: np.ndarray) -> Tuple[float, Dict[str, np.ndarray]]:
    """Mode-k mean cross-entropy and its gradient, canonical full-width form."""
    p = _vit.extract_dense(w, cfg, table, k)
    hd = cfg.dim // cfg.heads
    logits, cache = forward(p, images, hd, cfg.ln_eps)
    loss, dlogits = cross_entropy(logits, np.asarray(labels, dtype=np.int64))
    return loss, dense_to_canonical(backward(p, cache, dlogits, hd), cfg, table, k)


def growth_step(w: Dict[str, np.ndarray], cfg, table, k: int, images: np.ndarray,
                labels: np.ndarray, lr: float, clip: float) -> dict:
    """One growth step of mode k (k + 1 < num_modes).  Returns loss, the masked
    gradient G (.) grad, its L2 norm, the clip factor and the updated weights."""
    if not 0 <= k < table.num_modes - 1:
        raise ValueError("mode k needs a smaller mode k + 1 to grow from")
    ne = getattr(table, "n_embed", None)
    if ne is not None and int(ne[k]) != int(ne[k + 1]):
        raise ValueError("growth keeps the embedding width of modes k and k + 1")
    loss, grad = loss_and_grad(w, cfg, table, k, images, labels)
    G = growth_mask(cfg, table, k)
    gm = {key: G[key] * grad[key] for key in G}
    norm = math.sqrt(sum(float((a * a).sum()) for a in gm.values()))
    scale = 1.0 if norm <= clip else clip / norm
    new_w = {key: np.asarray(w[key], dtype=np.float64) - lr * scale * gm[key] for key in gm}
    return {"loss": loss, "masked_grad": gm, "norm": norm, "scale": scale, "weights": new_w,
            "mask": G}
