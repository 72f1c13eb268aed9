"""A textbook ViT forward built from torch CPU fp64 library ops (test helper).

Independent of the oracle: patch embedding is ``F.conv2d`` with stride P,
normalisation is ``F.layer_norm``, attention is
``F.scaled_dot_product_attention`` (default scale 1/sqrt(head_dim)) and the
activation is ``F.gelu(approximate='none')``.  Used only to pin the oracle.
"""
import contextlib

import numpy as np
import torch
import torch.nn.functional as F


def t64(a):
    if isinstance(a, torch.Tensor):
        return a
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def torch_vit(w, images, cfg, layer_heads=None, head_dim=None, grad=False):
    """Full-width (or per-layer ``layer_heads``) ViT over stacked canonical
    weights (or per-layer lists); ``head_dim`` defaults to dim / heads.  With
    ``grad`` the weights may be torch tensors that require gradients and the
    logits come back as a tensor of the autograd graph."""
    d, P, eps = cfg.dim, cfg.patch, cfg.ln_eps
    hd = head_dim or cfg.dim // cfg.heads
    with (contextlib.nullcontext() if grad else torch.no_grad()):
        x = F.conv2d(t64(images), t64(w["patch_w"]), t64(w["patch_b"]), stride=P)
        B = x.shape[0]
        x = x.flatten(2).transpose(1, 2)
        cls = t64(w["cls"]).reshape(1, 1, d).expand(B, 1, d)
        x = torch.cat([cls, x], dim=1) + t64(w["pos"])
        T = x.shape[1]
        for l in range(cfg.depth):
            u = F.layer_norm(x, (d,), t64(w["ln1_g"][l]), t64(w["ln1_b"][l]), eps)
            qkv_w = t64(w["qkv_w"][l])
            h = qkv_w.shape[0] // (3 * hd)
            qkv = F.linear(u, qkv_w, t64(w["qkv_b"][l])).reshape(B, T, 3, h, hd)
            q, k, v = qkv.permute(2, 0, 3, 1, 4).unbind(0)
            o = F.scaled_dot_product_attention(q, k, v)
            o = o.transpose(1, 2).reshape(B, T, h * hd)
            x = x + F.linear(o, t64(w["proj_w"][l]), t64(w["proj_b"][l]))
            u = F.layer_norm(x, (d,), t64(w["ln2_g"][l]), t64(w["ln2_b"][l]), eps)
            g = F.gelu(F.linear(u, t64(w["fc1_w"][l]), t64(w["fc1_b"][l])), approximate="none")
            x = x + F.linear(g, t64(w["fc2_w"][l]), t64(w["fc2_b"][l]))
        c = F.layer_norm(x[:, 0], (d,), t64(w["norm_g"]), t64(w["norm_b"]), eps)
        logits = F.linear(c, t64(w["head_w"]), t64(w["head_b"]))
        return logits if grad else logits.numpy()


def loop_masked_weights(w, cfg, table, k):
    """Zero pruned heads' q/k/v rows + proj columns and pruned units' fc1 rows +
    fc2 columns, one head / unit at a time (brute-force form of Eqs. 4 and 6)."""
    d, H, M = cfg.dim, cfg.heads, cfg.mlp_hidden
    hd = d // H
    out = {key: np.array(v, dtype=np.float64, copy=True) for key, v in w.items()}
    for l in range(cfg.depth):
        keep_h = set(int(i) for i in table.head_order[l][:table.n_heads[k][l]])
        keep_m = set(int(j) for j in table.mlp_order[l][:table.n_mlp[k][l]])
        for i in range(H):
            if i in keep_h:
                continue
            for t in range(3):
                for c in range(hd):
                    out["qkv_w"][l][t * d + i * hd + c, :] = 0.0
            for c in range(hd):
                out["proj_w"][l][:, i * hd + c] = 0.0
        for j in range(M):
            if j in keep_m:
                continue
            out["fc1_w"][l][j, :] = 0.0
            out["fc2_w"][l][:, j] = 0.0
    return out


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))


def loop_extract_embed(w, cfg, table, k):
    """Mode k as a smaller dense ViT, copied element by element: the active
    embedding channels (embed_order prefix), heads and MLP units.  Returns
    (weights with per-layer lists, active embedding width)."""
    d, H, M = cfg.dim, cfg.heads, cfg.mlp_hidden
    hd = d // H
    e = [int(c) for c in table.embed_order[:table.n_embed[k]]]
    E = len(e)
    out = {
        "patch_w": np.array([w["patch_w"][c] for c in e]),
        "patch_b": np.array([w["patch_b"][c] for c in e]),
        "cls": np.array([w["cls"][c] for c in e]),
        "pos": np.array([[w["pos"][t][c] for c in e] for t in range(w["pos"].shape[0])]),
        "norm_g": np.array([w["norm_g"][c] for c in e]),
        "norm_b": np.array([w["norm_b"][c] for c in e]),
        "head_w": np.array([[w["head_w"][n][c] for c in e] for n in range(w["head_w"].shape[0])]),
        "head_b": np.array(w["head_b"]),
    }
    for key in ("ln1_g", "ln1_b", "qkv_w", "qkv_b", "proj_w", "proj_b", "ln2_g", "ln2_b",
                "fc1_w", "fc1_b", "fc2_w", "fc2_b"):
        out[key] = []
    for l in range(cfg.depth):
        heads = [int(i) for i in table.head_order[l][:table.n_heads[k][l]]]
        units = [int(j) for j in table.mlp_order[l][:table.n_mlp[k][l]]]
        for key in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
            out[key].append(np.array([w[key][l][c] for c in e]))
        qrows = [t * d + i * hd + c2 for t in range(3) for i in heads for c2 in range(hd)]
        out["qkv_w"].append(np.array([[w["qkv_w"][l][r][c] for c in e] for r in qrows]))
        out["qkv_b"].append(np.array([w["qkv_b"][l][r] for r in qrows]))
        pcols = [i * hd + c2 for i in heads for c2 in range(hd)]
        out["proj_w"].append(np.array([[w["proj_w"][l][c][q] for q in pcols] for c in e]))
        out["proj_b"].append(np.array([w["proj_b"][l][c] for c in e]))
        out["fc1_w"].append(np.array([[w["fc1_w"][l][j][c] for c in e] for j in units]))
        out["fc1_b"].append(np.array([w["fc1_b"][l][j] for j in units]))
        out["fc2_w"].append(np.array([[w["fc2_w"][l][c][j] for j in units] for c in e]))
        out["fc2_b"].append(np.array([w["fc2_b"][l][c] for c in e]))
    return out, E
