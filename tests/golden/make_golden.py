"""Write the oracle's expected logits for the bf16 model configs.

Calls only the fp64 oracle (oracle/) on the seeded inputs
(paper_2609_10018_amd.inputs): the bf16-rounded matrices and images the
device holds, every DN mode, the full batch of each config (the first
GOLDEN_BATCH images where that table says so).  Logits are
computed in fp64 and stored as float32 (a relative rounding of 6e-8, far
below the 2e-2 bf16 tolerance they are compared at).

    python tests/golden/make_golden.py            # all bf16 configs (ViT and ResNet)
    python tests/golden/make_golden.py vit_ti     # one config
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from oracle import resnet as oracle_resnet  # noqa: E402
from paper_2609_10018_amd import inputs, inputs_cnn  # noqa: E402

OUT = os.path.dirname(os.path.abspath(__file__))
# Configs whose stored logits cover only the first images of the batch.
GOLDEN_BATCH = {"vit_b_emb": 16, "resnet50": 16}


def path_for(name: str) -> str:
    return os.path.join(OUT, f"logits_{name}.npz")


def make(name: str) -> None:
    cfg = inputs.CONFIGS[name]
    batch = GOLDEN_BATCH.get(name, cfg.batch)
    w = inputs.stored_weights(cfg, inputs.make_weights(cfg))
    x = inputs.stored_images(cfg, inputs.make_images(cfg, cfg.batch))[:batch]
    table = inputs.make_dn_table(cfg)
    out = np.zeros((table.num_modes, batch, cfg.num_classes), dtype=np.float32)
    for k in range(table.num_modes):
        t0 = time.time()
        out[k] = oracle.elastic_forward(w, cfg, table, k, x).astype(np.float32)
        print(f"{name} mode {k}: {time.time() - t0:.1f} s", flush=True)
    np.savez_compressed(path_for(name), logits=out, batch=batch,
                        numpy_version=np.__version__)


def make_cnn(name: str) -> None:
    """The elastic ResNet configs: same recipe (bf16-rounded filters and images)."""
    cfg = inputs_cnn.CNN_CONFIGS[name]
    batch = GOLDEN_BATCH.get(name, cfg.batch)
    w = inputs_cnn.stored_cnn_weights(cfg, inputs_cnn.make_cnn_weights(cfg))
    x = inputs.bf16_round(inputs_cnn.make_cnn_images(cfg, cfg.batch))[:batch]
    table = inputs_cnn.make_cnn_table(cfg)
    out = np.zeros((table.num_modes, batch, cfg.num_classes), dtype=np.float32)
    for k in range(table.num_modes):
        t0 = time.time()
        out[k] = oracle_resnet.elastic_forward(w, cfg, table, k, x).astype(np.float32)
        print(f"{name} mode {k}: {time.time() - t0:.1f} s", flush=True)
    np.savez_compressed(path_for(name), logits=out, batch=batch, numpy_version=np.__version__)


if __name__ == "__main__":
    names = sys.argv[1:] or ([n for n, c in inputs.CONFIGS.items() if c.dtype == inputs.BF16]
                             + list(inputs_cnn.CNN_CONFIGS))
    for n in names:
        make_cnn(n) if n in inputs_cnn.CNN_CONFIGS else make(n)
