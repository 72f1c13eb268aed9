"""fp64 CPU oracle for the elastic-ViT forward pass, the DN selection, the
growth step and the elastic ResNet forward.

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
CPU-baseline leg of bench.py, never by the product path.
"""
from .vit import (layer_norm, layer_norm_masked, gelu, softmax_rows, patchify, attention,
                  vit_forward, canonical_params, active_sets, active_embed, embed_mask, masks,
                  elastic_forward_masked, extract_dense, elastic_forward)
from .select import select_dn
from . import growth, resnet

__all__ = ["layer_norm", "layer_norm_masked", "active_embed", "embed_mask", "gelu", "softmax_rows", "patchify", "attention", "vit_forward",
           "canonical_params", "active_sets", "masks", "elastic_forward_masked",
           "extract_dense", "elastic_forward", "select_dn", "growth", "resnet"]
