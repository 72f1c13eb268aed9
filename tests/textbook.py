"""A textbook ViT forward built from torch CPU fp64 library ops (test helper).

Independent of the oracle: patch embedding is ``F.conv2d`` with stride P,
normalisation is ``F.layer_norm``, attention is
``F.scaled_dot_product_attention`` (default scale 1/sqrt(head_dim)) and the
activation is ``F.gelu(approximate='none')``.  Used only to pin the oracle.
"""
import numpy as np
import torch
import torch.nn.functional as F


def t64(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def torch_vit(w, images, cfg, layer_heads=None):
    """Full-width (or per-layer ``layer_heads``) ViT over stacked canonical weights."""
    d, P, hd, eps = cfg.dim, cfg.patch, cfg.dim // cfg.heads, cfg.ln_eps
    with torch.no_grad():
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
        return F.linear(c, t64(w["head_w"]), t64(w["head_b"])).numpy()


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
