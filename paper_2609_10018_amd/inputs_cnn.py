"""Seeded synthetic inputs for the elastic ResNet (bottleneck CNN) path.

Like ``inputs`` for the ViT, this module draws numbers and arranges them and
computes nothing that the forward pass computes.  It holds:

* bottleneck-ResNet shapes: ResNet-50 at 224x224 (stages of 3, 4, 6, 3 blocks,
  widths 64..512, expansion 4, the stride on the 3x3 convolution) and a small
  model of the same topology for fast checks;
* random-init weights in PyTorch order (convolutions [out, in, kh, kw]).  At
  inference a batch norm is a per-channel affine map, so every convolution
  here already carries it as its bias (folded form); He-normal filters keep
  activations in range through the depth, and each block's last convolution
  is scaled down (the usual small initial residual branch);
* DN tables: each bottleneck's two inner widths (outputs of its 1x1 reduce and
  of its 3x3 convolution) are elastic, as prefixes of one filter order per
  convolution (structured filter masks, Eq. 7; nested, Eq. 8), the filters
  ranked by saliency (mean absolute weight, most salient first).  The mode keep
  ratios are chosen so that the per-image MACs of ResNet-50's modes match the
  six DN levels the paper reports for it (Table 2).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

from .inputs import BF16, FP32, bf16_round, saliency_order  # noqa: F401  (shared dtype ids)

CNN_WEIGHT_SEED = 10
RESIDUAL_BRANCH_GAIN = 0.2


@dataclasses.dataclass(frozen=True)
class ResNetConfig:
    name: str
    img: int
    in_chans: int
    stem: int                       # stem output channels
    widths: Tuple[int, ...]         # bottleneck inner width per stage
    blocks: Tuple[int, ...]         # bottlenecks per stage
    expansion: int
    num_classes: int
    dtype: int
    batch: int

    def block_specs(self) -> List[dict]:
        """Per bottleneck: input channels, width, output channels, stride,
        input spatial size, and whether it has a projection shortcut."""
        out = []
        c_in = self.stem
        hw = self.img // 4                       # stride-2 stem, stride-2 max pool
        for s, (w, n) in enumerate(zip(self.widths, self.blocks)):
            for b in range(n):
                stride = 2 if (b == 0 and s > 0) else 1
                c_out = w * self.expansion
                out.append({"c_in": c_in, "width": w, "c_out": c_out, "stride": stride,
                            "hw_in": hw, "down": b == 0})
                hw = hw // stride
                c_in = c_out
        return out

    @property
    def features(self) -> int:
        return self.widths[-1] * self.expansion


CNN_CONFIGS: Dict[str, ResNetConfig] = {
    "resnet50": ResNetConfig("resnet50", 224, 3, 64, (64, 128, 256, 512), (3, 4, 6, 3), 4,
                             1000, BF16, 256),
    # Same topology (stride-2 stem and pool, four stages, stride on the 3x3),
    # narrower and shallower, 64x64 images: the oracle runs it in seconds.
    "resnet_small": ResNetConfig("resnet_small", 64, 3, 16, (16, 32, 64, 128), (1, 2, 2, 1), 4,
                                 100, BF16, 8),
}

# Per-mode keep ratio of the bottleneck widths (mode 0 = full; widths rounded
# to multiples of 8).  ResNet-50's ratios give 4.09, 3.35, 2.63, 2.02, 1.51
# and 1.08 GMACs per 224x224 image against the six DN levels of Table 2
# (4.12, 3.33, 2.65, 2.03, 1.51, 1.07 G).
CNN_MODE_RATIOS: Dict[str, List[float]] = {
    "resnet50": [1.0, 0.844, 0.695, 0.555, 0.407, 0.266],
    "resnet_small": [1.0, 0.75, 0.5, 0.25],
}


def conv_shapes(cfg: ResNetConfig) -> Dict[str, tuple]:
    """Canonical parameter names and shapes (convolutions [out, in, kh, kw])."""
    s = {"stem_w": (cfg.stem, cfg.in_chans, 7, 7), "stem_b": (cfg.stem,)}
    for i, b in enumerate(cfg.block_specs()):
        w, ci, co = b["width"], b["c_in"], b["c_out"]
        s[f"b{i}_c1_w"] = (w, ci, 1, 1)
        s[f"b{i}_c1_b"] = (w,)
        s[f"b{i}_c2_w"] = (w, w, 3, 3)
        s[f"b{i}_c2_b"] = (w,)
        s[f"b{i}_c3_w"] = (co, w, 1, 1)
        s[f"b{i}_c3_b"] = (co,)
        if b["down"]:
            s[f"b{i}_dn_w"] = (co, ci, 1, 1)
            s[f"b{i}_dn_b"] = (co,)
    s["fc_w"] = (cfg.num_classes, cfg.features)
    s["fc_b"] = (cfg.num_classes,)
    return s


def make_cnn_weights(cfg: ResNetConfig, seed: int = CNN_WEIGHT_SEED) -> Dict[str, np.ndarray]:
    """He-normal convolutions (std sqrt(2 / fan_in)), each block's last
    convolution times RESIDUAL_BRANCH_GAIN, biases N(0, 0.02^2), classifier
    N(0, 0.02^2); fp32, drawn tensor by tensor in conv_shapes order."""
    rng = np.random.default_rng(seed)
    w: Dict[str, np.ndarray] = {}
    for key, shp in conv_shapes(cfg).items():
        if key.endswith("_b"):
            a = rng.standard_normal(shp) * 0.02
        elif key == "fc_w":
            a = rng.standard_normal(shp) * 0.02
        else:
            fan_in = shp[1] * shp[2] * shp[3]
            a = rng.standard_normal(shp) * np.sqrt(2.0 / fan_in)
            if key.endswith("_c3_w"):
                a *= RESIDUAL_BRANCH_GAIN
        w[key] = a.astype(np.float32)
    return w


@dataclasses.dataclass
class CNNTable:
    """Per mode and bottleneck: active inner width (a prefix of each inner
    convolution's filter order)."""
    n_width: np.ndarray      # int32 [num_modes, num_blocks]
    order1: List[np.ndarray]  # per block: permutation of its width (1x1 reduce filters)
    order2: List[np.ndarray]  # per block: permutation of its width (3x3 filters)

    @property
    def num_modes(self) -> int:
        return int(self.n_width.shape[0])


def make_cnn_table(cfg: ResNetConfig, weights: Optional[Dict[str, np.ndarray]] = None) -> CNNTable:
    """Per-mode inner widths from CNN_MODE_RATIOS; each inner convolution's
    filters ordered by descending mean |w| of the filter (Eq. 7's filter
    saliency) of `weights` (default: the config's seeded weights)."""
    specs = cfg.block_specs()
    ratios = CNN_MODE_RATIOS[cfg.name]
    n = np.zeros((len(ratios), len(specs)), dtype=np.int32)
    for k, r in enumerate(ratios):
        for i, b in enumerate(specs):
            keep = int(np.floor(b["width"] * r / 8.0 + 0.5)) * 8
            n[k, i] = min(b["width"], max(8, keep))
    w = weights if weights is not None else make_cnn_weights(cfg)
    order1 = [saliency_order(w[f"b{i}_c1_w"]) for i in range(len(specs))]
    order2 = [saliency_order(w[f"b{i}_c2_w"]) for i in range(len(specs))]
    return CNNTable(n, order1, order2)


def stored_cnn_weights(cfg: ResNetConfig, w: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """The values the device holds: filters and classifier bf16-rounded on the
    bf16 path, biases fp32."""
    if cfg.dtype == FP32:
        return dict(w)
    return {k: (bf16_round(v) if k.endswith("_w") else v) for k, v in w.items()}


CNN_IMAGE_STATS_SEED = 5


def make_cnn_images(cfg: ResNetConfig, batch: int, seed: int = 1) -> np.ndarray:
    """fp32 NCHW images with per-image statistics: pixel (b, c, y, x) =
    offset[b, c] + contrast[b] * noise, noise N(0, 1) from `seed`, offsets
    N(0, 1) from CNN_IMAGE_STATS_SEED and contrasts U[0.25, 2] from the seed
    after it.  Like
    normalised natural images, images differ in channel means and contrast;
    white noise alone reaches the pooled features of a random network almost
    only through its batch-common part."""
    rng = np.random.default_rng(seed)
    noise = rng.standard_normal((batch, cfg.in_chans, cfg.img, cfg.img), dtype=np.float64)
    # One generator per statistic, so that the first b images of a batch do
    # not depend on the batch size.
    offset = np.random.default_rng(CNN_IMAGE_STATS_SEED).standard_normal(
        (batch, cfg.in_chans, 1, 1))
    contrast = np.random.default_rng(CNN_IMAGE_STATS_SEED + 1).uniform(0.25, 2.0, (batch, 1, 1, 1))
    return (offset + contrast * noise).astype(np.float32)
