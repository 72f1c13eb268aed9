"""Helpers shared by the GPU tests: device tensors from numpy, the error
metric (max |error| over the whole logits array / max |expected|) and the
top-1 agreement."""
import numpy as np
import torch

from paper_2609_10018_amd import inputs

# Top-1 agreement is required on the rows whose expected top-2 gap exceeds
# TIE_BAND x max|expected|.  A bf16 forward cannot order two logits closer
# than about one rounding unit of the largest one (2^-8 = 3.9e-3 relative);
# the band is that, rounded up, and a quarter of the 2e-2 error bar, so a
# row can flip only within it.  The band is fixed in advance, not derived
# from the errors a run measures.
TIE_BAND = 5e-3
# At most this fraction of the rows may fall inside the band, so the check
# cannot pass by excluding most of them.  With random-init weights and 1000
# classes the expected top-2 gaps are small (the oracle logits put 0-28% of a
# config's rows inside the band, per mode; small batches of 16-32 images
# scatter most).
MAX_TIED_FRACTION = 1.0 / 3.0


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


def top1_agreement(got: np.ndarray, ref: np.ndarray, band: float = TIE_BAND) -> dict:
    """Top-1 agreement of `got` with `ref` (rows = images).

    raw: fraction of rows whose argmax agrees.  decisive: the same over the
    rows whose expected top-2 gap ref[c1] - ref[c2] exceeds band * max|ref|
    (n_decisive of them); flips: (row, gap / max|ref|, the row's max |error|
    / max|ref|) of every disagreeing row."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = float(np.max(np.abs(ref)))
    g, r = np.argmax(got, axis=1), np.argmax(ref, axis=1)
    top2 = np.sort(ref, axis=1)[:, -2:]
    gap = (top2[:, 1] - top2[:, 0]) / scale
    decisive = gap > band
    agree = g == r
    row_err = np.max(np.abs(got - ref), axis=1) / scale
    return {
        "raw": float(np.mean(agree)),
        "decisive": float(np.mean(agree[decisive])) if decisive.any() else 1.0,
        "n_decisive": int(decisive.sum()),
        "n": int(ref.shape[0]),
        "flips": [(int(i), float(gap[i]), float(row_err[i])) for i in np.flatnonzero(~agree)],
    }


def check_top1(label: str, got: np.ndarray, ref: np.ndarray, minimum: float = 0.995) -> dict:
    """Print the agreement and assert it: decisive agreement >= minimum and at
    most MAX_TIED_FRACTION of the rows inside the tie band."""
    a = top1_agreement(got, ref)
    print(f"{label}: top-1 raw {a['raw']:.4f}, decisive {a['decisive']:.4f} "
          f"({a['n_decisive']}/{a['n']} rows outside the {TIE_BAND:g} band), flips "
          + ", ".join(f"row {i} gap {gp:.2e} err {e:.2e}" for i, gp, e in a["flips"]))
    assert a["n_decisive"] >= (1.0 - MAX_TIED_FRACTION) * a["n"], a
    assert a["decisive"] >= minimum, a
    return a
