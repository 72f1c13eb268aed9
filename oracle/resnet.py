"""Plain fp64 CPU oracle for the elastic bottleneck-ResNet forward pass.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run anything in this package.
It shares no code with the HIP path and imports nothing from it.

What it computes: a ResNet-50-style network at inference (the paper's CNN
backbone, Section 4.1 and Table 2): a 7x7 stride-2 stem convolution with ReLU,
3x3 stride-2 max pooling, bottleneck blocks (1x1 reduce, 3x3 with the block's
stride, 1x1 expand; a 1x1 projection shortcut with the same stride on each
stage's first block; ReLU after the sum), global average pooling and a linear
classifier.  Batch norm at inference is a per-channel affine map and is carried
in each convolution's bias.

A DN keeps a subset of each bottleneck's inner filters.  Eq. 7 masks whole
kernels of a convolution; a pruned filter of the 1x1 reduce removes its output
channel and the matching input channels of the 3x3, a pruned 3x3 filter its
output channel and the matching input channels of the 1x1 expand.  Three
formulations, as for the ViT:

* ``resnet_forward``         (F1) a dense network whose inner widths may be any;
* ``elastic_forward_masked`` (F2) full-width filters times the {0,1} kernel
                              masks of Eq. 7, then F1;
* ``extract_dense``          (F3) copies mode k's active filters into a
                              narrower dense network, which F1 then runs.

Parity status: pinned in tests/test_oracle_cnn.py by torch CPU fp64 library
ops (F.conv2d, F.max_pool2d, adaptive average pooling, F.linear), brute-force
convolution and pooling loops, mask form vs gather form and locality.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np


def conv2d(x: np.ndarray, w: np.ndarray, b: np.ndarray, stride: int, pad: int) -> np.ndarray:
    """x [N, C, H, W], w [O, C, KH, KW] -> [N, O, Ho, Wo] (cross-correlation,
    zero padding), as one matmul over explicitly gathered patches."""
    N, C, H, W = x.shape
    O, _, KH, KW = w.shape
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (W + 2 * pad - KW) // stride + 1
    cols = np.empty((N, Ho, Wo, C, KH, KW), dtype=np.float64)
    for i in range(KH):
        for j in range(KW):
            cols[:, :, :, :, i, j] = xp[:, :, i:i + stride * Ho:stride,
                                        j:j + stride * Wo:stride].transpose(0, 2, 3, 1)
    y = cols.reshape(N * Ho * Wo, C * KH * KW) @ w.reshape(O, -1).T + b
    return y.reshape(N, Ho, Wo, O).transpose(0, 3, 1, 2)


def max_pool_3x3_s2(x: np.ndarray) -> np.ndarray:
    """3x3 window, stride 2, padding 1 (padding never wins the max)."""
    N, C, H, W = x.shape
    xp = np.pad(x, ((0, 0), (0, 0), (1, 1), (1, 1)), constant_values=-np.inf)
    Ho, Wo = (H - 1) // 2 + 1, (W - 1) // 2 + 1
    out = np.full((N, C, Ho, Wo), -np.inf)
    for i in range(3):
        for j in range(3):
            out = np.maximum(out, xp[:, :, i:i + 2 * Ho:2, j:j + 2 * Wo:2])
    return out


def relu(x: np.ndarray) -> np.ndarray:
    return np.maximum(x, 0.0)


def canonical_params(w: Dict[str, np.ndarray], cfg) -> dict:
    """Flat canonical arrays -> F1's nested form, fp64."""
    f = lambda a: np.asarray(a, dtype=np.float64)
    p = {"stem": (f(w["stem_w"]), f(w["stem_b"])), "fc": (f(w["fc_w"]), f(w["fc_b"])),
         "blocks": []}
    for i, spec in enumerate(cfg.block_specs()):
        blk = {"stride": spec["stride"]}
        for c in ("c1", "c2", "c3", "dn"):
            if f"b{i}_{c}_w" in w:
                blk[c] = (f(w[f"b{i}_{c}_w"]), f(w[f"b{i}_{c}_b"]))
        p["blocks"].append(blk)
    return p


def resnet_forward(p: dict, images: np.ndarray) -> np.ndarray:
    """F1: dense bottleneck-ResNet forward in fp64; logits [N, classes]."""
    x = relu(conv2d(np.asarray(images, dtype=np.float64), *p["stem"], stride=2, pad=3))
    x = max_pool_3x3_s2(x)
    for blk in p["blocks"]:
        s = blk["stride"]
        y = relu(conv2d(x, *blk["c1"], stride=1, pad=0))
        y = relu(conv2d(y, *blk["c2"], stride=s, pad=1))
        y = conv2d(y, *blk["c3"], stride=1, pad=0)
        short = conv2d(x, *blk["dn"], stride=s, pad=0) if "dn" in blk else x
        x = relu(y + short)
    feat = x.mean(axis=(2, 3))
    return feat @ p["fc"][0].T + p["fc"][1]


def active_filters(table, k: int, block: int):
    """Active filters of mode k in one block: (1x1 reduce, 3x3), in order."""
    n = int(table.n_width[k][block])
    return (np.asarray(table.order1[block][:n], dtype=np.int64),
            np.asarray(table.order2[block][:n], dtype=np.int64))


def elastic_forward_masked(w: Dict[str, np.ndarray], cfg, table, k: int,
                           images: np.ndarray) -> np.ndarray:
    """F2: Eq. 7 kernel masks on the full-width filters (a pruned filter's
    kernels and bias, and the input kernels that read its channel, are zero),
    then F1."""
    p = canonical_params(w, cfg)
    for i, blk in enumerate(p["blocks"]):
        a1, a2 = active_filters(table, k, i)
        m1 = np.zeros(blk["c1"][0].shape[0])
        m1[a1] = 1.0
        m2 = np.zeros(blk["c2"][0].shape[0])
        m2[a2] = 1.0
        w1, b1 = blk["c1"]
        w2, b2 = blk["c2"]
        w3, b3 = blk["c3"]
        blk["c1"] = (w1 * m1[:, None, None, None], b1 * m1)
        blk["c2"] = (w2 * m2[:, None, None, None] * m1[None, :, None, None], b2 * m2)
        blk["c3"] = (w3 * m2[None, :, None, None], b3)
    return resnet_forward(p, images)


def extract_dense(w: Dict[str, np.ndarray], cfg, table, k: int) -> dict:
    """F3: copy mode k's active filters, in order, into a narrower network."""
    p = canonical_params(w, cfg)
    for i, blk in enumerate(p["blocks"]):
        a1, a2 = active_filters(table, k, i)
        w1, b1 = blk["c1"]
        w2, b2 = blk["c2"]
        w3, b3 = blk["c3"]
        blk["c1"] = (w1[a1].copy(), b1[a1].copy())
        blk["c2"] = (w2[a2][:, a1].copy(), b2[a2].copy())
        blk["c3"] = (w3[:, a2].copy(), b3)
    return p


def elastic_forward(w: Dict[str, np.ndarray], cfg, table, k: int, images: np.ndarray,
                    chunk: int = 8) -> np.ndarray:
    """Mode-k logits via F3 + F1, in image chunks."""
    p = extract_dense(w, cfg, table, k)
    outs: List[np.ndarray] = []
    for s in range(0, images.shape[0], chunk):
        outs.append(resnet_forward(p, images[s:s + chunk]))
    return np.concatenate(outs, axis=0)
