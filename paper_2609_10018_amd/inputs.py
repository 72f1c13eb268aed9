"""Seeded synthetic inputs shared by the HIP path's tests/bench and the oracle.

This module draws numbers and arranges them; it computes nothing that the
elastic forward pass computes.  It holds:

* the four model shapes (a tiny fp32 model and ViT-Ti/S/B-shaped bf16 models,
  patch 16 at 224x224 for the latter three, ViT-B as in the paper's
  experimental setup section),
* random-init weights in the canonical PyTorch ``[out, in]`` order,
* N(0, 1) images in NCHW (a stand-in for normalised ImageNet images; no
  dataset is used),
* the Descendant-Network (DN) tables: one channel order per layer and, per
  mode, how many heads / MLP units of that order are active.  Nested DNs
  (weight sharing, Eq. 8) make every mode a prefix of one order.
* round-to-nearest-even fp32 -> bf16 rounding of host arrays, so the oracle
  can be fed exactly the values the bf16 path stores.

The channel order is the paper's saliency order (Section 4.1, Eq. 4): rows
ranked by their average absolute weight, most salient first, applied to the
seeded weights.  Building a DN table is the design-time pruning step, not a
step of the forward: the table is input data to the HIP path and to the
oracle alike, and neither of them ranks anything.
"""
from __future__ import annotations

import dataclasses
import functools
from typing import Dict, List, Optional

import numpy as np

FP32 = 0
BF16 = 1

WEIGHT_SEED = 0
IMAGE_SEED = 1
RATIO_SEED = 2
SEQUENCE_SEED = 3
INIT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    img: int
    patch: int
    in_chans: int
    dim: int
    depth: int
    heads: int
    mlp_hidden: int
    num_classes: int
    dtype: int
    batch: int
    ln_eps: float = 1e-6

    @property
    def grid(self) -> int:
        return self.img // self.patch

    @property
    def num_patches(self) -> int:
        return self.grid * self.grid

    @property
    def tokens(self) -> int:
        return self.num_patches + 1

    @property
    def head_dim(self) -> int:
        return self.dim // self.heads

    @property
    def patch_k(self) -> int:
        return self.in_chans * self.patch * self.patch


CONFIGS: Dict[str, ModelConfig] = {
    # 32x32x3, patch 8 -> 16 patches + CLS, d 64, 2 layers, 2 heads, MLP 128, 10 classes.
    "tiny": ModelConfig("tiny", 32, 8, 3, 64, 2, 2, 128, 10, FP32, 4),
    "vit_ti": ModelConfig("vit_ti", 224, 16, 3, 192, 12, 3, 768, 1000, BF16, 64),
    "vit_s": ModelConfig("vit_s", 224, 16, 3, 384, 12, 6, 1536, 1000, BF16, 128),
    "vit_b": ModelConfig("vit_b", 224, 16, 3, 768, 12, 12, 3072, 1000, BF16, 256),
    # Same shapes with modes that also narrow the embedding width.
    "tiny_emb": ModelConfig("tiny_emb", 32, 8, 3, 64, 2, 2, 128, 10, FP32, 4),
    "vit_ti_emb": ModelConfig("vit_ti_emb", 224, 16, 3, 192, 12, 3, 768, 1000, BF16, 32),
    "vit_b_emb": ModelConfig("vit_b_emb", 224, 16, 3, 768, 12, 12, 3072, 1000, BF16, 256),
}

# Per-mode (heads, MLP hidden[, embedding width]) caps; mode 0 is full width,
# larger k is smaller.  Without a third entry every mode keeps all d channels.
MODE_CAPS: Dict[str, List[tuple]] = {
    "tiny": [(2, 128), (1, 64)],
    "vit_ti": [(3, 768), (2, 576), (1, 384), (1, 192)],
    "vit_s": [(6, 1536), (5, 1152), (4, 768), (3, 384), (2, 230)],
    "vit_b": [(12, 3072), (9, 2304), (6, 1536), (3, 768), (2, 460)],
    "tiny_emb": [(2, 128, 64), (2, 96, 48), (1, 64, 24)],
    "vit_ti_emb": [(3, 768, 192), (2, 576, 144), (1, 384, 96), (1, 192, 64)],
    "vit_b_emb": [(12, 3072, 768), (9, 2304, 576), (6, 1536, 384), (3, 768, 192)],
}
# Configs whose per-layer widths follow a per-layer keep ratio r_l ~ U[0.15, 1].
LAYER_RATIO_CONFIGS = ("vit_s",)

# Canonical per-layer parameter names, in draw order.
LAYER_KEYS = ("ln1_g", "ln1_b", "qkv_w", "qkv_b", "proj_w", "proj_b",
              "ln2_g", "ln2_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")
# Matrices stored in bf16 by the bf16 path (vectors stay fp32).
MATRIX_KEYS = ("patch_w", "qkv_w", "proj_w", "fc1_w", "fc2_w", "head_w")


def param_shapes(cfg: ModelConfig) -> Dict[str, tuple]:
    d, T, M, C = cfg.dim, cfg.tokens, cfg.mlp_hidden, cfg.num_classes
    s = {"patch_w": (d, cfg.in_chans, cfg.patch, cfg.patch), "patch_b": (d,),
         "cls": (d,), "pos": (T, d)}
    layer = {"ln1_g": (d,), "ln1_b": (d,), "qkv_w": (3 * d, d), "qkv_b": (3 * d,),
             "proj_w": (d, d), "proj_b": (d,), "ln2_g": (d,), "ln2_b": (d,),
             "fc1_w": (M, d), "fc1_b": (M,), "fc2_w": (d, M), "fc2_b": (d,)}
    for key, shp in layer.items():
        s[key] = (cfg.depth,) + shp
    s.update({"norm_g": (d,), "norm_b": (d,), "head_w": (C, d), "head_b": (C,)})
    return s


def param_count(cfg: ModelConfig) -> int:
    return int(sum(np.prod(v) for v in param_shapes(cfg).values()))


def make_weights(cfg: ModelConfig, seed: int = WEIGHT_SEED) -> Dict[str, np.ndarray]:
    """Random-init weights, fp32, canonical order; per-layer arrays stacked on axis 0.

    Every tensor is N(0, 0.02^2) except LayerNorm scales, which are
    1 + N(0, 0.02^2), so that no branch is scaled away and biases are non-zero.
    Draws happen tensor by tensor (layer by layer for stacked ones).
    """
    rng = np.random.default_rng(seed)
    shapes = param_shapes(cfg)

    def draw(shape, gain_one=False):
        a = rng.standard_normal(shape, dtype=np.float64) * INIT_STD
        if gain_one:
            a += 1.0
        return a.astype(np.float32)

    w: Dict[str, np.ndarray] = {}
    for key in ("patch_w", "patch_b", "cls", "pos"):
        w[key] = draw(shapes[key])
    per_layer = {k: [] for k in LAYER_KEYS}
    for _ in range(cfg.depth):
        for key in LAYER_KEYS:
            per_layer[key].append(draw(shapes[key][1:], gain_one=key.endswith("_g")))
    for key in LAYER_KEYS:
        w[key] = np.ascontiguousarray(np.stack(per_layer[key]))
    w["norm_g"] = draw(shapes["norm_g"], gain_one=True)
    w["norm_b"] = draw(shapes["norm_b"])
    w["head_w"] = draw(shapes["head_w"])
    w["head_b"] = draw(shapes["head_b"])
    return w


def make_images(cfg: ModelConfig, batch: int, seed: int = IMAGE_SEED) -> np.ndarray:
    """N(0, 1) pixels, fp32, NCHW [batch, 3, img, img]."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((batch, cfg.in_chans, cfg.img, cfg.img),
                               dtype=np.float64).astype(np.float32)


def layer_ratios(cfg: ModelConfig, seed: int = RATIO_SEED) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.uniform(0.15, 1.0, size=cfg.depth)


@dataclasses.dataclass
class DNTable:
    """Per-layer channel orders and per-mode active counts (prefix lengths)."""
    n_heads: np.ndarray      # int32 [num_modes, depth]
    n_mlp: np.ndarray        # int32 [num_modes, depth]
    head_order: np.ndarray   # int32 [depth, heads], a permutation per layer
    mlp_order: np.ndarray    # int32 [depth, mlp_hidden], a permutation per layer
    n_embed: Optional[np.ndarray] = None      # int32 [num_modes]; None: all d channels
    embed_order: Optional[np.ndarray] = None  # int32 [dim], shared by all layers; None: identity

    @property
    def num_modes(self) -> int:
        return int(self.n_heads.shape[0])

    @property
    def depth(self) -> int:
        return int(self.n_heads.shape[1])


def saliency_order(rows: np.ndarray) -> np.ndarray:
    """Indices of the rows of `rows` ([n, ...]) by descending mean |value|
    (Eq. 4's L1 row saliency); equal scores keep the lower index first."""
    score = np.abs(np.asarray(rows, dtype=np.float64)).reshape(rows.shape[0], -1).mean(axis=1)
    return np.argsort(-score, kind="stable").astype(np.int32)


def _orders(cfg: ModelConfig, w: Dict[str, np.ndarray]):
    d, hd, L = cfg.dim, cfg.head_dim, cfg.depth
    # qkv_w rows t*d + i*hd + c (t = q, k, v) belong to head i.
    head_order = np.stack([
        saliency_order(w["qkv_w"][l].reshape(3, cfg.heads, hd, d).transpose(1, 0, 2, 3))
        for l in range(L)])
    mlp_order = np.stack([saliency_order(w["fc1_w"][l]) for l in range(L)])
    return head_order, mlp_order, saliency_order(w["patch_w"])


@functools.lru_cache(maxsize=None)
def _seeded_orders(cfg: ModelConfig):
    out = _orders(cfg, make_weights(cfg))
    for a in out:
        a.setflags(write=False)
    return out


def make_dn_table(cfg: ModelConfig, weights: Optional[Dict[str, np.ndarray]] = None) -> DNTable:
    """DN table of a config: per-mode widths from MODE_CAPS (per-layer ratios
    for LAYER_RATIO_CONFIGS) and per-layer channel orders by saliency of
    `weights` (default: the config's seeded weights):
    * heads: the mean |w| over the head's q, k and v rows of qkv_w;
    * MLP units: the mean |w| of the unit's fc1_w row;
    * embedding channels (one order for every layer): the mean |w| of the
      channel's patch-embedding row."""
    caps = MODE_CAPS[cfg.name]
    L = cfg.depth
    n_heads = np.zeros((len(caps), L), dtype=np.int32)
    n_mlp = np.zeros((len(caps), L), dtype=np.int32)
    ratios = layer_ratios(cfg) if cfg.name in LAYER_RATIO_CONFIGS else None
    for k, cap in enumerate(caps):
        hk, mk = cap[0], cap[1]
        for l in range(L):
            if ratios is None or k == 0:
                n_heads[k, l], n_mlp[k, l] = hk, mk
            else:
                n_heads[k, l] = max(1, int(np.floor(hk * ratios[l] + 0.5)))
                n_mlp[k, l] = max(1, int(np.floor(mk * ratios[l] + 0.5)))
    head_order, mlp_order, embed_order = (_orders(cfg, weights) if weights is not None
                                          else _seeded_orders(cfg))
    n_embed = np.array([cap[2] if len(cap) > 2 else cfg.dim for cap in caps], dtype=np.int32)
    return DNTable(n_heads, n_mlp, head_order, mlp_order, n_embed, embed_order)


def mode_sequence(n: int, num_modes: int, seed: int = SEQUENCE_SEED) -> np.ndarray:
    """Seeded random sequence of mode indices for the latency regime."""
    return np.random.default_rng(seed).integers(0, num_modes, size=n).astype(np.int32)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32 holding them."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out.reshape(a.shape)


def stored_weights(cfg: ModelConfig, w: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """The values the device holds: matrices bf16-rounded on the bf16 path, vectors fp32."""
    if cfg.dtype == FP32:
        return dict(w)
    return {k: (bf16_round(v) if k in MATRIX_KEYS else v) for k, v in w.items()}


def stored_images(cfg: ModelConfig, x: np.ndarray) -> np.ndarray:
    return x if cfg.dtype == FP32 else bf16_round(x)
