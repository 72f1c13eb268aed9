"""ctypes binding of the C ABI in include/elasto.h (argument marshalling only).

Every computation runs in the HIP library; this module converts numpy host
arrays and torch device tensors into the plain pointers and sizes the C ABI
takes, and turns status codes into exceptions.  If the library is not built
this module raises: there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Dict, Optional

import numpy as np

from .inputs import BF16, FP32, DNTable, ModelConfig

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libelasto.so")

c_i32, c_i64, c_f32, c_f64, c_vp = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                     ctypes.c_double, ctypes.c_void_p)

STATUS = {0: "OK", 1: "INVALID_ARG", 2: "BAD_CONFIG", 3: "BAD_TABLE", 4: "OUT_OF_MEMORY",
          5: "HIP", 6: "MODE_RANGE", 7: "BATCH_RANGE", 8: "INFEASIBLE"}

# Tensor ids (elasto_tensor_t).
T_PATCH_W, T_PATCH_B, T_CLS, T_POS, T_NORM_G, T_NORM_B, T_HEAD_W, T_HEAD_B = range(8)
(T_LN1_G, T_LN1_B, T_WQKV, T_BQKV, T_WO, T_BO, T_LN2_G, T_LN2_B, T_W1, T_B1, T_W2,
 T_B2) = range(8, 20)
# Kernel classes (elasto_kernel_t).
KERNELS = ["patch", "ln", "qkv", "attn", "proj", "fc1", "fc2", "head"]
# Epilogues (elasto_epilogue_t).
EPI_BIAS, EPI_BIAS_GELU, EPI_BIAS_RESID, EPI_BIAS_F32OUT = range(4)

WEIGHT_FIELDS = ["patch_w", "patch_b", "cls", "pos", "ln1_g", "ln1_b", "qkv_w", "qkv_b",
                 "proj_w", "proj_b", "ln2_g", "ln2_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b",
                 "norm_g", "norm_b", "head_w", "head_b"]


class ElastoError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"elasto {STATUS.get(status, status)}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [(n, c_i32) for n in ("img", "patch", "in_chans", "dim", "depth", "heads",
                                     "mlp_hidden", "num_classes", "max_batch", "dtype")] + \
               [("ln_eps", c_f32)]


class Weights(ctypes.Structure):
    _fields_ = [(n, c_vp) for n in WEIGHT_FIELDS]


class Table(ctypes.Structure):
    _fields_ = [("num_modes", c_i32), ("depth", c_i32), ("n_heads", c_vp), ("n_mlp", c_vp),
                ("head_order", c_vp), ("mlp_order", c_vp), ("n_embed", c_vp),
                ("embed_order", c_vp)]


class DNLut(ctypes.Structure):
    _fields_ = [("num_modes", c_i32), ("flops", ctypes.POINTER(c_f64)),
                ("latency_ms", ctypes.POINTER(c_f64)), ("memory_bytes", ctypes.POINTER(c_f64)),
                ("accuracy", ctypes.POINTER(c_f64)), ("power_w", ctypes.POINTER(c_f64))]


class CNNConfig(ctypes.Structure):
    _fields_ = [("img", c_i32), ("in_chans", c_i32), ("stem", c_i32), ("num_stages", c_i32),
                ("widths", c_i32 * 8), ("blocks", c_i32 * 8), ("expansion", c_i32),
                ("num_classes", c_i32), ("max_batch", c_i32), ("dtype", c_i32)]


class CNNWeights(ctypes.Structure):
    _fields_ = [("num_tensors", c_i32), ("tensors", ctypes.POINTER(ctypes.c_void_p))]


class CNNTableC(ctypes.Structure):
    _fields_ = [("num_modes", c_i32), ("num_blocks", c_i32), ("n_width", c_vp),
                ("order1", c_vp), ("order2", c_vp)]


_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() or "
                          f"python -m paper_2609_10018_amd.build")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    sig = {
        "elasto_create": [P(Config), P(Weights), P(Table), P(c_vp)],
        "elasto_destroy": [c_vp],
        "elasto_set_mode": [c_vp, c_i32],
        "elasto_get_mode": [c_vp, P(c_i32)],
        "elasto_forward": [c_vp, c_vp, c_i32, c_vp, c_vp],
        "elasto_forward_static": [c_vp, c_vp, c_i32, c_vp, c_vp],
        "elasto_mode_info": [c_vp, c_i32, P(c_f64), P(c_i64)],
        "elasto_memory_info": [c_vp, P(c_i64), P(c_i64)],
        "elasto_validate": [P(Config), P(Table)],
        "elasto_packed_bytes": [P(Config), P(c_i64)],
        "elasto_packed_layout": [P(Config), c_i32, c_i32, P(c_i64), P(c_i64), P(c_i64), P(c_i32)],
        "elasto_pack_weights": [P(Config), P(Weights), P(Table), c_vp, c_i64],
        "elasto_kernel_timing": [c_vp, c_i32, c_i32],
        "elasto_kernel_timing_read": [c_vp, P(c_f64), P(c_i64)],
        "elasto_kernel_work": [c_vp, c_i32, c_i32, c_i32, P(c_f64), P(c_f64), P(c_i32)],
        "elasto_op_layernorm": [c_i32, c_vp, c_i64, c_vp, c_i32, c_vp, c_i64, c_i32, c_vp, c_vp,
                                c_f32, c_vp],
        "elasto_op_linear": [c_i32, c_i32, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i32,
                             c_vp, c_i64, c_i32, c_i32, c_vp],
        "elasto_op_linear_ln": [c_i32, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i32, c_vp,
                                c_i64, c_i32, c_i32, c_vp, c_vp, c_i64, c_vp, c_f32, c_vp],
        "elasto_op_attention": [c_i32, c_vp, c_i64, c_vp, c_i64, c_i32, c_i32, c_i32, c_i32,
                                c_f32, c_vp],
        "elasto_op_conv2d": [c_vp, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32,
                             c_vp, c_i64, c_i64, c_vp, c_vp, c_i64, c_i32, c_i32, c_vp],
        "elasto_select_mode": [P(DNLut), c_f64, c_f64, c_f64, c_f64, P(c_i32)],
        "elasto_growth_create": [c_vp, c_i32, P(c_vp)],
        "elasto_growth_destroy": [c_vp],
        "elasto_growth_step": [c_vp, c_i32, c_vp, c_vp, c_i32, c_f32, c_f32, c_vp, c_vp],
        "elasto_growth_read": [c_vp, c_i32, c_vp, c_i64],
        "elasto_profile_modes": [c_vp, c_vp, c_i32, c_vp, c_i32, c_i32, c_vp, P(c_f64), P(c_f64),
                                 P(c_f64)],
        "elasto_cnn_validate": [P(CNNConfig), P(CNNTableC)],
        "elasto_cnn_create": [P(CNNConfig), P(CNNWeights), P(CNNTableC), P(c_vp)],
        "elasto_cnn_destroy": [c_vp],
        "elasto_cnn_set_mode": [c_vp, c_i32],
        "elasto_cnn_get_mode": [c_vp, P(c_i32)],
        "elasto_cnn_forward": [c_vp, c_vp, c_i32, c_vp, c_vp],
        "elasto_cnn_mode_info": [c_vp, c_i32, P(c_f64), P(c_i64)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = c_i32
    lib.elasto_last_error.argtypes = []
    lib.elasto_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def last_error() -> str:
    return load_library().elasto_last_error().decode()


def check(status: int) -> None:
    if status != 0:
        raise ElastoError(status, last_error())


def make_config(cfg: ModelConfig, max_batch: int) -> Config:
    return Config(cfg.img, cfg.patch, cfg.in_chans, cfg.dim, cfg.depth, cfg.heads,
                  cfg.mlp_hidden, cfg.num_classes, max_batch, cfg.dtype, cfg.ln_eps)


class _HostWeights:
    """Keeps contiguous fp32 copies alive while the C struct points at them."""

    def __init__(self, w: Dict[str, np.ndarray]):
        self.arrays = {k: np.ascontiguousarray(w[k], dtype=np.float32) for k in WEIGHT_FIELDS}
        self.struct = Weights(*[a.ctypes.data for a in (self.arrays[k] for k in WEIGHT_FIELDS)])


class _HostTable:
    """Keeps int32 copies alive while the C struct points at them; the
    embedding columns are optional (None: every mode keeps all channels,
    identity order)."""

    def __init__(self, t: DNTable):
        cols = (t.n_heads, t.n_mlp, t.head_order, t.mlp_order,
                getattr(t, "n_embed", None), getattr(t, "embed_order", None))
        self.arrays = [None if a is None else np.ascontiguousarray(a, dtype=np.int32)
                       for a in cols]
        self.struct = Table(int(t.n_heads.shape[0]), int(t.n_heads.shape[1]),
                            *[None if a is None else a.ctypes.data for a in self.arrays])


def validate(cfg: ModelConfig, table: DNTable, max_batch: int = 1) -> int:
    c = make_config(cfg, max_batch)
    t = _HostTable(table)
    return load_library().elasto_validate(ctypes.byref(c), ctypes.byref(t.struct))


def packed_bytes(cfg: ModelConfig) -> int:
    out = c_i64()
    check(load_library().elasto_packed_bytes(ctypes.byref(make_config(cfg, 1)), ctypes.byref(out)))
    return out.value


def packed_layout(cfg: ModelConfig, tensor: int, layer: int = 0):
    off, rows, cols, eb = c_i64(), c_i64(), c_i64(), c_i32()
    check(load_library().elasto_packed_layout(ctypes.byref(make_config(cfg, 1)), tensor, layer,
                                              ctypes.byref(off), ctypes.byref(rows),
                                              ctypes.byref(cols), ctypes.byref(eb)))
    return off.value, rows.value, cols.value, eb.value


def pack_weights(cfg: ModelConfig, w: Dict[str, np.ndarray], table: DNTable) -> np.ndarray:
    n = packed_bytes(cfg)
    dst = np.zeros(n, dtype=np.uint8)
    hw, ht = _HostWeights(w), _HostTable(table)
    check(load_library().elasto_pack_weights(ctypes.byref(make_config(cfg, 1)),
                                             ctypes.byref(hw.struct), ctypes.byref(ht.struct),
                                             dst.ctypes.data, n))
    return dst


def _stream_ptr(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return int(getattr(stream, "cuda_stream", stream))


class ElasticViT:
    """One library handle: packed weights on the current device + scratch."""

    def __init__(self, cfg: ModelConfig, w: Dict[str, np.ndarray], table: DNTable,
                 max_batch: int):
        self.lib = load_library()
        self.cfg = cfg
        self.max_batch = max_batch
        self.num_modes = int(table.n_heads.shape[0])
        c = make_config(cfg, max_batch)
        hw, ht = _HostWeights(w), _HostTable(table)
        h = c_vp()
        check(self.lib.elasto_create(ctypes.byref(c), ctypes.byref(hw.struct),
                                     ctypes.byref(ht.struct), ctypes.byref(h)))
        self.h = h

    def close(self) -> None:
        if getattr(self, "h", None) is not None and self.h.value:
            check(self.lib.elasto_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_mode(self, k: int) -> None:
        check(self.lib.elasto_set_mode(self.h, int(k)))

    def get_mode(self) -> int:
        k = c_i32()
        check(self.lib.elasto_get_mode(self.h, ctypes.byref(k)))
        return k.value

    def forward(self, images, logits, stream=None) -> None:
        """images: device tensor NCHW (bf16 or fp32 per the path); logits: fp32 device tensor."""
        if not images.is_contiguous() or not logits.is_contiguous():
            raise ValueError("images and logits must be contiguous")
        check(self.lib.elasto_forward(self.h, images.data_ptr(), int(images.shape[0]),
                                      logits.data_ptr(), _stream_ptr(stream)))

    def forward_static(self, images, logits, stream=None) -> None:
        """The forward with its activations in the library's static scratch
        (elasto_forward_static: allocates nothing)."""
        if not images.is_contiguous() or not logits.is_contiguous():
            raise ValueError("images and logits must be contiguous")
        check(self.lib.elasto_forward_static(self.h, images.data_ptr(), int(images.shape[0]),
                                             logits.data_ptr(), _stream_ptr(stream)))

    def mode_info(self, k: int):
        f, b = c_f64(), c_i64()
        check(self.lib.elasto_mode_info(self.h, int(k), ctypes.byref(f), ctypes.byref(b)))
        return f.value, b.value

    def profile_modes(self, images, logits, warmup: int = 3, iters: int = 10, stream=None):
        """Per-mode (latency_ms, memory_bytes, flops) arrays at images.shape[0]."""
        n = self.num_modes
        lat, mem, fl = (np.zeros(n, dtype=np.float64) for _ in range(3))
        dp = ctypes.POINTER(c_f64)
        check(self.lib.elasto_profile_modes(
            self.h, images.data_ptr(), int(images.shape[0]), logits.data_ptr(), int(warmup),
            int(iters), _stream_ptr(stream), lat.ctypes.data_as(dp), mem.ctypes.data_as(dp),
            fl.ctypes.data_as(dp)))
        return lat, mem, fl

    def memory_info(self):
        wb, sb = c_i64(), c_i64()
        check(self.lib.elasto_memory_info(self.h, ctypes.byref(wb), ctypes.byref(sb)))
        return wb.value, sb.value

    def kernel_timing(self, kernel: str, max_launches: int) -> None:
        kc = -1 if kernel is None else KERNELS.index(kernel)
        check(self.lib.elasto_kernel_timing(self.h, kc, int(max_launches)))

    def kernel_timing_read(self):
        ms, n = c_f64(), c_i64()
        check(self.lib.elasto_kernel_timing_read(self.h, ctypes.byref(ms), ctypes.byref(n)))
        return ms.value, n.value

    def kernel_work(self, k: int, batch: int, kernel: str):
        f, b, n = c_f64(), c_f64(), c_i32()
        check(self.lib.elasto_kernel_work(self.h, int(k), int(batch), KERNELS.index(kernel),
                                          ctypes.byref(f), ctypes.byref(b), ctypes.byref(n)))
        return f.value, b.value, n.value


def _ptr(t):
    return None if t is None else t.data_ptr()


def op_layernorm(dtype: int, x, x_stride: int, out, rows: int, d: int, g, b, eps: float,
                 x_cls=None, tokens: int = 1, stream=None) -> None:
    check(load_library().elasto_op_layernorm(dtype, x.data_ptr(), x_stride, _ptr(x_cls), tokens,
                                             out.data_ptr(), rows, d, g.data_ptr(), b.data_ptr(),
                                             eps, _stream_ptr(stream)))


def op_linear(dtype: int, epilogue: int, A, lda: int, W, ldw: int, C, ldc: int, bias,
              M: int, N: int, K: int, C_cls=None, tokens: int = 1, stream=None) -> None:
    check(load_library().elasto_op_linear(dtype, epilogue, A.data_ptr(), lda, W.data_ptr(), ldw,
                                          C.data_ptr(), ldc, _ptr(C_cls), tokens, bias.data_ptr(),
                                          M, N, K, _stream_ptr(stream)))


def op_linear_ln(epilogue: int, A, lda: int, W, ldw: int, C, ldc: int, bias, M: int, N: int,
                 K: int, stats_ld: int, stats_out=None, stats_in=None, colsum=None,
                 eps: float = 1e-6, C_cls=None, tokens: int = 1, stream=None) -> None:
    check(load_library().elasto_op_linear_ln(epilogue, A.data_ptr(), lda, W.data_ptr(), ldw,
                                             C.data_ptr(), ldc, _ptr(C_cls), tokens,
                                             bias.data_ptr(), M, N, K, _ptr(stats_out),
                                             _ptr(stats_in), stats_ld, _ptr(colsum), eps,
                                             _stream_ptr(stream)))


def op_attention(dtype: int, qkv, qkv_stride: int, o, o_stride: int, batch: int, tokens: int,
                 heads: int, head_dim: int, scale: float, stream=None) -> None:
    check(load_library().elasto_op_attention(dtype, qkv.data_ptr(), qkv_stride, o.data_ptr(),
                                             o_stride, batch, tokens, heads, head_dim, scale,
                                             _stream_ptr(stream)))


class GrowthContext:
    """Growth-step state of a bf16 ElasticViT handle (fp32 masters, saved
    activations, gradients) for batches of up to max_batch images."""

    def __init__(self, vit: "ElasticViT", max_batch: int):
        self.lib = load_library()
        self.vit = vit                      # the handle must outlive the context
        g = c_vp()
        check(self.lib.elasto_growth_create(vit.h, int(max_batch), ctypes.byref(g)))
        self.g = g

    def step(self, mode: int, images, labels, lr: float, clip: float, stats=None,
             stream=None) -> None:
        """images: bf16 device tensor NCHW; labels: int32 device tensor [batch];
        stats: fp32 device tensor with 3 elements (loss, |G grad|, clip factor) or None."""
        if not images.is_contiguous() or not labels.is_contiguous():
            raise ValueError("images and labels must be contiguous")
        check(self.lib.elasto_growth_step(self.g, int(mode), images.data_ptr(), labels.data_ptr(),
                                          int(images.shape[0]), float(lr), float(clip),
                                          _ptr(stats), _stream_ptr(stream)))

    def read(self, which: int) -> np.ndarray:
        """which 0: packed weights (uint8); 1: fp32 masters (float32, one per bf16 element)."""
        total = packed_bytes(self.vit.cfg)
        n = total if which == 0 else total // 2 * 4
        buf = np.empty(n, dtype=np.uint8)
        check(self.lib.elasto_growth_read(self.g, int(which), buf.ctypes.data, n))
        return buf if which == 0 else buf.view(np.float32)

    def close(self) -> None:
        if getattr(self, "g", None) is not None and self.g.value:
            check(self.lib.elasto_growth_destroy(self.g))
            self.g = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def op_conv2d(x, batch: int, H: int, W: int, cs: int, ca: int, kh: int, kw: int, stride: int,
              pad: int, w, ldw: int, wseg: int, bias, y, ldy: int, n: int, relu: bool = False,
              stream=None) -> None:
    check(load_library().elasto_op_conv2d(x.data_ptr(), batch, H, W, cs, ca, kh, kw, stride, pad,
                                          w.data_ptr(), ldw, wseg, bias.data_ptr(), y.data_ptr(),
                                          ldy, n, int(relu), _stream_ptr(stream)))


class _HostCNN:
    """Keeps the host arrays alive while the C structs point at them."""

    def __init__(self, cfg, w, table, max_batch: int):
        from .inputs_cnn import conv_shapes
        self.cfg = CNNConfig()
        self.cfg.img, self.cfg.in_chans, self.cfg.stem = cfg.img, cfg.in_chans, cfg.stem
        self.cfg.num_stages = len(cfg.widths)
        for i, (wd, nb) in enumerate(zip(cfg.widths, cfg.blocks)):
            self.cfg.widths[i], self.cfg.blocks[i] = wd, nb
        self.cfg.expansion, self.cfg.num_classes = cfg.expansion, cfg.num_classes
        self.cfg.max_batch, self.cfg.dtype = max_batch, cfg.dtype
        self.tensors = [] if w is None else [
            np.ascontiguousarray(w[key], dtype=np.float32) for key in conv_shapes(cfg)]
        self.ptrs = (ctypes.c_void_p * max(1, len(self.tensors)))(
            *[t.ctypes.data for t in self.tensors])
        self.weights = CNNWeights(len(self.tensors), self.ptrs)
        self.n_width = np.ascontiguousarray(table.n_width, dtype=np.int32)
        self.order1 = np.ascontiguousarray(np.concatenate(table.order1), dtype=np.int32)
        self.order2 = np.ascontiguousarray(np.concatenate(table.order2), dtype=np.int32)
        self.table = CNNTableC(int(self.n_width.shape[0]), int(self.n_width.shape[1]),
                               self.n_width.ctypes.data, self.order1.ctypes.data,
                               self.order2.ctypes.data)


def cnn_validate(cfg, table, max_batch: int = 1) -> int:
    hc = _HostCNN(cfg, None, table, max_batch)
    return load_library().elasto_cnn_validate(ctypes.byref(hc.cfg), ctypes.byref(hc.table))


class ElasticResNet:
    """One elastic bottleneck-ResNet handle (bf16, NHWC on the device)."""

    def __init__(self, cfg, w, table, max_batch: int):
        self.lib = load_library()
        self.cfg = cfg
        self.num_modes = int(table.n_width.shape[0])
        hc = _HostCNN(cfg, w, table, max_batch)
        h = c_vp()
        check(self.lib.elasto_cnn_create(ctypes.byref(hc.cfg), ctypes.byref(hc.weights),
                                         ctypes.byref(hc.table), ctypes.byref(h)))
        self.h = h

    def close(self) -> None:
        if getattr(self, "h", None) is not None and self.h.value:
            check(self.lib.elasto_cnn_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_mode(self, k: int) -> None:
        check(self.lib.elasto_cnn_set_mode(self.h, int(k)))

    def get_mode(self) -> int:
        k = c_i32()
        check(self.lib.elasto_cnn_get_mode(self.h, ctypes.byref(k)))
        return k.value

    def forward(self, images, logits, stream=None) -> None:
        check(self.lib.elasto_cnn_forward(self.h, images.data_ptr(), int(images.shape[0]),
                                          logits.data_ptr(), _stream_ptr(stream)))

    def mode_info(self, k: int):
        f, b = c_f64(), c_i64()
        check(self.lib.elasto_cnn_mode_info(self.h, int(k), ctypes.byref(f), ctypes.byref(b)))
        return f.value, b.value


def select_mode(flops, latency_ms, memory_bytes, accuracy=None, power_w=None,
                max_latency_ms=math.inf, max_memory_bytes=math.inf, min_accuracy=-math.inf,
                max_power_w=math.inf):
    """Eq. 11 over a DN table (host only).  Returns the mode, or None when no
    mode meets the bounds."""
    cols = [np.ascontiguousarray(c, dtype=np.float64) if c is not None else None
            for c in (flops, latency_ms, memory_bytes, accuracy, power_w)]
    n = len(cols[0])
    if any(c is not None and len(c) != n for c in cols):
        raise ValueError("table columns differ in length")
    dp = ctypes.POINTER(c_f64)
    ptr = [c.ctypes.data_as(dp) if c is not None else None for c in cols]
    lut = DNLut(n, *ptr)
    k = c_i32(-1)
    st = load_library().elasto_select_mode(ctypes.byref(lut), float(max_latency_ms),
                                           float(max_memory_bytes), float(min_accuracy),
                                           float(max_power_w), ctypes.byref(k))
    if st == 8:
        return None
    check(st)
    return k.value


__all__ = ["ElasticViT", "ElasticResNet", "cnn_validate", "select_mode", "ElastoError", "load_library", "validate", "packed_bytes",
           "packed_layout", "pack_weights", "op_layernorm", "op_linear", "op_linear_ln", "op_attention",
           "KERNELS", "FP32", "BF16"]
