"""Helpers shared by the GPU tests: device tensors from numpy, the R11 error
metric and the tie-aware top-1 agreement."""
import numpy as np
import torch

from paper_2609_10018_amd import inputs


def dev(a: np.ndarray, dtype) -> torch.Tensor:
    """numpy -> device tensor; bf16 conversion rounds to nearest even."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(dtype).cuda().contiguous()


def images_on_device(cfg, x: np.ndarray) -> torch.Tensor:
    return dev(x, torch.bfloat16 if cfg.dtype == inputs.BF16 else torch.float32)


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max |got - ref| over the whole array / max |ref|."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))


def top1_agreement(got: np.ndarray, ref: np.ndarray, tie_rel: float = 2e-2):
    """(raw, tie_aware) fraction of rows whose argmax agrees.  A row whose GPU
    argmax c' has ref[c*] - ref[c'] <= tie_rel * max|ref| counts as agreeing in
    the tie-aware figure (several answers are correct within the tolerance)."""
    g = np.argmax(got, axis=1)
    r = np.argmax(ref, axis=1)
    raw = float(np.mean(g == r))
    scale = np.max(np.abs(ref))
    gap = ref[np.arange(ref.shape[0]), r] - ref[np.arange(ref.shape[0]), g]
    tie = float(np.mean((g == r) | (gap <= tie_rel * scale)))
    return raw, tie
