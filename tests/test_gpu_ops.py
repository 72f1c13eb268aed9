"""Kernel-level parity: each HIP kernel (through the C ABI's single-kernel
entry points) against the oracle's fp64 pieces on the same inputs."""
import math

import numpy as np
import pytest

import oracle
from oracle import resnet as orn
from paper_2609_10018_amd import ffi, inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gpu_util import dev, rel_err  # noqa: E402

BF16, FP32 = inputs.BF16, inputs.FP32


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ffi.load_library()


@pytest.mark.parametrize("dtype,rows,d", [(BF16, 1000, 768), (BF16, 197, 192), (BF16, 5, 384),
                                          (BF16, 9, 2048), (BF16, 3, 8),
                                          (FP32, 68, 64), (FP32, 300, 200)])
def test_layernorm(dtype, rows, d):
    rng = np.random.default_rng(rows + d)
    x = (rng.standard_normal((rows, d)) * 2 + 0.5).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    b = (0.1 * rng.standard_normal(d)).astype(np.float32)
    tdt = torch.bfloat16 if dtype == BF16 else torch.float32
    xd = dev(x, tdt)
    out = torch.empty((rows, d), dtype=tdt, device="cuda")
    gd, bd = dev(g, torch.float32), dev(b, torch.float32)
    ffi.op_layernorm(dtype, xd, d, out, rows, d, gd, bd, 1e-6)
    torch.cuda.synchronize()
    ref = oracle.layer_norm(host(xd), g.astype(np.float64), b.astype(np.float64), 1e-6)
    tol = 8e-3 if dtype == BF16 else 2e-6
    assert rel_err(host(out), ref) < tol


def test_layernorm_strided_rows():
    rng = np.random.default_rng(1)
    T, d, B = 197, 768, 4
    x = rng.standard_normal((B * T, d)).astype(np.float32)
    xd = dev(x, torch.bfloat16)
    out = torch.empty((B, d), dtype=torch.bfloat16, device="cuda")
    g = dev(np.ones(d), torch.float32)
    b = dev(np.zeros(d), torch.float32)
    ffi.op_layernorm(BF16, xd, T * d, out, B, d, g, b, 1e-6)
    torch.cuda.synchronize()
    ref = oracle.layer_norm(host(xd)[::T], np.ones(d), np.zeros(d), 1e-6)
    assert rel_err(host(out), ref) < 8e-3


@pytest.mark.parametrize("tokens", [197, 1])
def test_layernorm_fp32_class_rows(tokens):
    """bf16 rows, with every tokens-th row read as fp32 from the class-row buffer."""
    rng = np.random.default_rng(2)
    B, d = 5, 768
    rows = B * tokens
    x = rng.standard_normal((rows, d)).astype(np.float32)
    xc = (rng.standard_normal((B, d)) * 1e-3 + 0.25).astype(np.float32)  # needs fp32 precision
    xd, xcd = dev(x, torch.bfloat16), dev(xc, torch.float32)
    g = dev(1 + 0.1 * rng.standard_normal(d), torch.float32)
    b = dev(0.1 * rng.standard_normal(d), torch.float32)
    out = torch.empty((rows, d), dtype=torch.bfloat16, device="cuda")
    ffi.op_layernorm(BF16, xd, d, out, rows, d, g, b, 1e-6, x_cls=xcd, tokens=tokens)
    torch.cuda.synchronize()
    xin = host(xd)
    xin[::tokens] = xc.astype(np.float64)
    ref = oracle.layer_norm(xin, host(g), host(b), 1e-6)
    assert rel_err(host(out), ref) < 8e-3


def _linear_case(dtype, epi, M, N, K, lda, ldw, ldc, poison=False, seed=0, tokens=0):
    rng = np.random.default_rng(seed)
    tdt = torch.bfloat16 if dtype == BF16 else torch.float32
    A = rng.standard_normal((M, lda)).astype(np.float32)
    W = (rng.standard_normal((N + 7, ldw)) * 0.05).astype(np.float32)
    if poison:
        A[:, K:] = np.nan
        W[:, K:] = np.nan
        W[N:, :] = np.nan
    bias = (0.1 * rng.standard_normal(N)).astype(np.float32)
    C0 = rng.standard_normal((M, ldc)).astype(np.float32)
    Ad, Wd = dev(A, tdt), dev(W, tdt)
    Cd = dev(C0, torch.float32 if epi == ffi.EPI_BIAS_F32OUT else tdt)
    C_before = host(Cd)
    ccls = None
    if tokens:
        ccls = dev(rng.standard_normal((M // tokens, N)) * 1e-3 + 0.5, torch.float32)
        ccls_before = host(ccls)
    ffi.op_linear(dtype, epi, Ad, lda, Wd, ldw, Cd, ldc, dev(bias, torch.float32), M, N, K,
                  C_cls=ccls, tokens=max(tokens, 1))
    torch.cuda.synchronize()
    a64, w64 = host(Ad)[:, :K], host(Wd)[:N, :K]
    z = a64 @ w64.T + bias.astype(np.float64)
    if epi == ffi.EPI_BIAS_GELU:
        z = oracle.gelu(z)
    elif epi == ffi.EPI_BIAS_RESID:
        base = C_before[:, :N].copy()
        if tokens:
            base[::tokens] = ccls_before
        z = base + z
    got = host(Cd)
    if tokens:
        np.testing.assert_array_equal(got[::tokens], C_before[::tokens])  # class rows untouched in C
        got[::tokens, :N] = host(ccls)
    return got[:, :N], z, got[:, N:], C_before[:, N:]


LINEAR_CASES = [
    # dtype, epilogue, M, N, K, lda, ldw, ldc
    (BF16, ffi.EPI_BIAS, 1000, 2304, 768, 768, 768, 2304),
    (BF16, ffi.EPI_BIAS_GELU, 777, 460, 768, 768, 768, 3072),
    (BF16, ffi.EPI_BIAS_RESID, 513, 768, 460, 3072, 3072, 768),
    (BF16, ffi.EPI_BIAS_RESID, 300, 384, 230, 1536, 1536, 384),
    (BF16, ffi.EPI_BIAS_F32OUT, 256, 1000, 768, 768, 768, 1000),
    (BF16, ffi.EPI_BIAS, 33, 192, 64, 192, 192, 576),
    (BF16, ffi.EPI_BIAS, 1, 8, 8, 8, 8, 8),
    # enough 256x256 tiles for a second, 128x256-tile launch over the last rows
    (BF16, ffi.EPI_BIAS_GELU, 21999, 3072, 768, 768, 768, 3072),
    (BF16, ffi.EPI_BIAS_RESID, 22000, 768, 3072, 3072, 3072, 768),
    # persistent 256x256 kernel (Bias / BiasGelu): one partial round with
    # ragged rows; several tiles per CU with ragged rows; ragged N with ldc > N
    (BF16, ffi.EPI_BIAS, 7000, 2304, 768, 768, 768, 2304),
    (BF16, ffi.EPI_BIAS, 20000, 2304, 768, 768, 768, 2304),
    (BF16, ffi.EPI_BIAS_GELU, 12800, 1272, 384, 384, 384, 1280),
    (BF16, ffi.EPI_BIAS_RESID, 12800, 1272, 384, 384, 384, 1280),
    (BF16, ffi.EPI_BIAS_RESID, 30000, 768, 1024, 1024, 1024, 768),
    # fewer 128x128 tiles than CUs: 4-stage load pipeline (48 K steps; exactly 4)
    (BF16, ffi.EPI_BIAS_RESID, 400, 768, 3072, 3072, 3072, 768),
    (BF16, ffi.EPI_BIAS, 500, 512, 256, 256, 256, 512),
    # outputs at most 64 wide: 256x64 tiles
    (BF16, ffi.EPI_BIAS, 3001, 64, 256, 256, 256, 64),
    (BF16, ffi.EPI_BIAS_RESID, 777, 40, 576, 576, 576, 48),
    (FP32, ffi.EPI_BIAS, 68, 192, 64, 64, 64, 192),
    (FP32, ffi.EPI_BIAS_GELU, 70, 67, 61, 64, 61, 128),
    (FP32, ffi.EPI_BIAS_RESID, 68, 64, 33, 64, 128, 64),
    (FP32, ffi.EPI_BIAS_F32OUT, 4, 10, 64, 64, 64, 10),
]


@pytest.mark.parametrize("case", LINEAR_CASES, ids=[f"{c[0]}-{c[1]}-{c[2]}x{c[3]}x{c[4]}" for c in LINEAR_CASES])
def test_linear(case):
    dtype, epi, M, N, K, lda, ldw, ldc = case
    got, ref, tail_after, tail_before = _linear_case(dtype, epi, M, N, K, lda, ldw, ldc)
    tol = 1e-2 if dtype == BF16 else 1e-5
    assert rel_err(got, ref) < tol
    np.testing.assert_array_equal(tail_after, tail_before)  # columns >= N untouched


@pytest.mark.parametrize("images", [4, 112])
def test_linear_residual_fp32_class_rows(images):
    """The bf16 residual epilogue keeps class-token rows in the fp32 side buffer
    (112 images: the rows are split over two launches of different tiles)."""
    got, ref, tail_after, tail_before = _linear_case(BF16, ffi.EPI_BIAS_RESID, images * 197, 768,
                                                     460, 3072, 3072, 768, tokens=197)
    assert rel_err(got, ref) < 1e-2
    cls_err = np.abs(got[::197] - ref[::197]).max() / np.abs(ref[::197]).max()
    assert cls_err < 1e-5      # fp32 rows: no bf16 rounding of the class rows
    np.testing.assert_array_equal(tail_after, tail_before)


@pytest.mark.parametrize("dtype", [BF16, FP32])
def test_linear_reads_no_inactive_weights(dtype):
    """NaN beyond the K prefix (A and W) and beyond the N rows of W never leaks."""
    got, ref, _, _ = _linear_case(dtype, ffi.EPI_BIAS_RESID, 300, 460, 460, 512, 3072, 768,
                                  poison=True)
    assert np.isfinite(got).all()
    assert rel_err(got, ref) < (1e-2 if dtype == BF16 else 1e-5)


def _attention_ref(qkv, B, T, h, hd, scale):
    out = np.zeros((B * T, h * hd))
    for b in range(B):
        for s in range(h):
            blk = qkv[b * T:(b + 1) * T, s * 3 * hd:(s + 1) * 3 * hd]
            q, k, v = blk[:, :hd], blk[:, hd:2 * hd], blk[:, 2 * hd:]
            p = oracle.softmax_rows(q @ k.T * scale)
            out[b * T:(b + 1) * T, s * hd:(s + 1) * hd] = p @ v
    return out


@pytest.mark.parametrize("dtype,B,T,h,hd,stride", [
    (BF16, 3, 197, 5, 64, 2304),
    (BF16, 2, 197, 1, 64, 576),
    (BF16, 2, 17, 2, 64, 384),
    (BF16, 1, 240, 3, 64, 576),
    (BF16, 2, 1, 2, 64, 384),
    # the last key tile exactly full: one tile, an even and an odd tile count
    (BF16, 3, 16, 2, 64, 384),
    (BF16, 2, 32, 3, 64, 576),
    (BF16, 2, 224, 2, 64, 384),
    # more (sequence, head) pairs than workgroups: each walks several pairs
    (BF16, 100, 197, 3, 64, 576),
    (BF16, 130, 33, 4, 64, 768),
    (FP32, 4, 17, 2, 32, 192),
    (FP32, 2, 197, 3, 64, 576),
])
def test_attention(dtype, B, T, h, hd, stride):
    rng = np.random.default_rng(T + h)
    qkv = (rng.standard_normal((B * T, stride)) * 1.5).astype(np.float32)
    tdt = torch.bfloat16 if dtype == BF16 else torch.float32
    qd = dev(qkv, tdt)
    o_stride = stride // 3
    od = torch.zeros((B * T, o_stride), dtype=tdt, device="cuda")
    scale = 1.0 / math.sqrt(hd)
    ffi.op_attention(dtype, qd, stride, od, o_stride, B, T, h, hd, scale)
    torch.cuda.synchronize()
    ref = _attention_ref(host(qd), B, T, h, hd, scale)
    got = host(od)[:, :h * hd]
    assert rel_err(got, ref) < (2e-2 if dtype == BF16 else 1e-5)
    assert (host(od)[:, h * hd:] == 0).all()


# Implicit-GEMM convolution (elastic ResNet layers) against the oracle's fp64
# conv2d.  Cases: ragged output width and rows, a channel prefix (ca < cs),
# several 64-channel steps per tap, odd image sizes with stride 2, a
# non-square kernel, the smallest channel count, enough 256x256 tiles for the
# split launch, and channel counts of at most 32 (taps sharing a K step).
CONV_CASES = [
    # batch, H, W, cs, ca, kh, kw, stride, pad, wseg, n, ldy, relu
    (3, 14, 14, 64, 56, 3, 3, 1, 1, 64, 40, 48, True),
    (2, 15, 15, 128, 128, 3, 3, 2, 1, 136, 72, 72, False),
    (2, 28, 28, 256, 256, 1, 1, 2, 0, 256, 512, 512, False),
    (1, 5, 5, 16, 8, 3, 3, 1, 1, 8, 8, 8, True),
    (2, 9, 13, 32, 24, 3, 1, 1, 1, 32, 16, 16, False),
    (85, 28, 28, 64, 64, 3, 3, 1, 1, 64, 256, 256, True),
    # at most 32 active channels: several taps share one 64-wide K step
    (4, 56, 56, 64, 16, 3, 3, 2, 1, 64, 16, 16, True),
    (2, 14, 14, 64, 32, 3, 3, 1, 1, 64, 32, 32, True),
    (3, 7, 7, 24, 24, 3, 3, 1, 1, 24, 24, 24, False),
]


def _conv_case(batch, H, W, cs, ca, kh, kw, stride, pad, wseg, n, ldy, relu, seed=5,
               poison=False):
    rng = np.random.default_rng(seed)
    x = inputs.bf16_round(rng.standard_normal((batch, H, W, cs)))
    w = inputs.bf16_round(rng.standard_normal((n, kh * kw, wseg)) / math.sqrt(kh * kw * ca))
    b = rng.standard_normal(n).astype(np.float32) * 0.1
    y0 = inputs.bf16_round(rng.standard_normal((batch * ((H + 2 * pad - kh) // stride + 1) *
                                                ((W + 2 * pad - kw) // stride + 1), ldy)))
    if poison:  # what the kernel must never read
        x[..., ca:] = np.nan
        w[:, :, ca:] = np.nan
    xd, wd, yd = dev(x, torch.bfloat16), dev(w.reshape(n, -1), torch.bfloat16), dev(y0, torch.bfloat16)
    ffi.op_conv2d(xd, batch, H, W, cs, ca, kh, kw, stride, pad, wd, kh * kw * wseg, wseg,
                  dev(b, torch.float32), yd, ldy, n, relu)
    torch.cuda.synchronize()
    got = host(yd)
    x_nchw = np.nan_to_num(x[..., :ca]).transpose(0, 3, 1, 2)
    w_oihw = np.nan_to_num(w[:, :, :ca]).reshape(n, kh, kw, ca).transpose(0, 3, 1, 2)
    ref = orn.conv2d(x_nchw, w_oihw, b.astype(np.float64), stride, pad)
    ref = ref.transpose(0, 2, 3, 1).reshape(-1, n)
    if relu:
        ref = np.maximum(ref, 0.0)
    return got[:, :n], ref, got[:, n:], y0[:, n:]


@pytest.mark.parametrize("case", CONV_CASES, ids=[f"b{c[0]}-{c[1]}x{c[2]}-c{c[4]}of{c[3]}-"
                                                  f"k{c[5]}x{c[6]}s{c[7]}-n{c[10]}" for c in CONV_CASES])
def test_conv2d(case):
    got, ref, tail_after, tail_before = _conv_case(*case)
    assert rel_err(got, ref) < 1e-2
    np.testing.assert_array_equal(tail_after, tail_before)  # columns >= n untouched


def test_conv2d_never_reads_inactive_channels():
    case = CONV_CASES[0]
    clean, ref, _, _ = _conv_case(*case)
    poisoned, _, _, _ = _conv_case(*case, poison=True)
    assert np.isfinite(poisoned).all()
    np.testing.assert_array_equal(poisoned, clean)
    assert rel_err(clean, ref) < 1e-2
