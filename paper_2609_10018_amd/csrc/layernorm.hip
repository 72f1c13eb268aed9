// LayerNorm over the feature axis: u = (x - mean) / sqrt(var + eps) * g + b,
// biased variance, statistics in fp32.  Memory-bound: each lane holds its
// share of a row in registers (two passes over registers, one read of the row
// from HBM, one write).
//
// The bf16 path gives each row half a wave and reads and writes 16-byte
// (8-element) bf16 vectors; the class-token rows of the residual stream are
// fp32 and come from their own buffer.  Row stride is free.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

constexpr int kMaxChunks = 8;  // 8-element chunks per lane: d <= 2048

__device__ __forceinline__ float half_sum(float v) {
#pragma unroll
  for (int off = 16; off >= 1; off >>= 1) v += __shfl_xor(v, off, 32);
  return v;
}

// Two rows per wave (32 lanes each), so a load instruction moves 16 bytes per
// lane; NC = ceil(d / 256) chunks per lane.  Rows past the end re-read the
// last row and store nothing.
template <int NC>
__global__ __launch_bounds__(256) void layernorm_bf16_kernel(const uint16_t* __restrict__ x,
                                                             int64_t x_stride,
                                                             const float* __restrict__ xcls,
                                                             int tokens,
                                                             uint16_t* __restrict__ out,
                                                             int64_t rows, int d,
                                                             const float* __restrict__ g,
                                                             const float* __restrict__ b,
                                                             float eps) {
  const int hl = threadIdx.x & 31;
  const int64_t row_raw = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 5);
  const bool live = row_raw < rows;
  const int64_t row = live ? row_raw : rows - 1;
  const int nch = d >> 3;
  const int64_t bi = xcls != nullptr ? row / tokens : 0;
  const bool cls_row = xcls != nullptr && row == bi * tokens;  // uniform per half-wave
  const uint16_t* xr = x + row * x_stride;
  const float* xc = cls_row ? xcls + bi * (int64_t)d : nullptr;
  float v[NC][8];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int ci = hl + 32 * i;
    if (ci < nch) {
      if (cls_row) {
        const f32x4 w0 = *reinterpret_cast<const f32x4*>(xc + 8 * ci);
        const f32x4 w1 = *reinterpret_cast<const f32x4*>(xc + 8 * ci + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[i][e] = w0[e];
          v[i][4 + e] = w1[e];
        }
      } else {
        const u32x4 w = *reinterpret_cast<const u32x4*>(xr + 8 * ci);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[i][2 * e] = __uint_as_float(w[e] << 16);
          v[i][2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[i][e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[i][e] = 0.0f;
    }
  }
  const float inv_d = 1.0f / (float)d;
  const float mean = half_sum(s) * inv_d;
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    if (hl + 32 * i < nch) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float c = v[i][e] - mean;
        ss += c * c;
      }
    }
  }
  const float rstd = rsqrtf(half_sum(ss) * inv_d + eps);
  if (!live) return;
  uint16_t* orow = out + row * (int64_t)d;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int ci = hl + 32 * i;
    if (ci < nch) {
      const f32x4 g0 = *reinterpret_cast<const f32x4*>(g + 8 * ci);
      const f32x4 g1 = *reinterpret_cast<const f32x4*>(g + 8 * ci + 4);
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(b + 8 * ci);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(b + 8 * ci + 4);
      const float gv[8] = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
      const float bv[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w[e] = pack_bf16x2((v[i][2 * e] - mean) * rstd * gv[2 * e] + bv[2 * e],
                           (v[i][2 * e + 1] - mean) * rstd * gv[2 * e + 1] + bv[2 * e + 1]);
      }
      *reinterpret_cast<u32x4*>(orow + 8 * ci) = w;
    }
  }
}

// fp32 rows, any d <= 2048 (element-wise access).
__global__ __launch_bounds__(256) void layernorm_f32_kernel(const float* __restrict__ x,
                                                            int64_t x_stride,
                                                            float* __restrict__ out, int64_t rows,
                                                            int d, const float* __restrict__ g,
                                                            const float* __restrict__ b,
                                                            float eps) {
  constexpr int kMax = 32;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float* xr = x + row * x_stride;
  float v[kMax];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    v[i] = c < d ? xr[c] : 0.0f;
    s += v[i];
  }
  const float mean = wave_sum(s) / (float)d;
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    if (c < d) ss += (v[i] - mean) * (v[i] - mean);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(ss) / (float)d + eps);
  float* orow = out + row * (int64_t)d;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    if (c < d) orow[c] = (v[i] - mean) * rstd * g[c] + b[c];
  }
}

template <int NC>
hipError_t launch_ln(const uint16_t* x, int64_t x_stride, const float* xcls, int tokens,
                     uint16_t* out, int64_t rows, int d, const float* g, const float* b, float eps,
                     hipStream_t s) {
  hipLaunchKernelGGL(layernorm_bf16_kernel<NC>, dim3((unsigned)((rows + 7) / 8)), dim3(256), 0, s,
                     x, x_stride, xcls, tokens, out, rows, d, g, b, eps);
  return hipGetLastError();
}

// Weights of a LayerNorm folded into the following linear layer: one wave
// per output row n.  Sums over the row accumulate in fp64 (the folded column
// sum is of the bf16-rounded products the GEMM multiplies).
constexpr int kFoldMaxWidths = 16;
struct FoldWidths {
  int n;
  int e[kFoldMaxWidths];
};

__global__ __launch_bounds__(256) void ln_fold_kernel(const uint16_t* __restrict__ W, int N, int D,
                                                      const float* __restrict__ gamma,
                                                      const float* __restrict__ beta,
                                                      const float* __restrict__ bias,
                                                      FoldWidths wd, uint16_t* __restrict__ Wf,
                                                      float* __restrict__ colsum,
                                                      float* __restrict__ cbias, int64_t ldv) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const uint16_t* w = W + (int64_t)n * D;
  uint16_t* wf = Wf + (int64_t)n * D;
  double sw[kFoldMaxWidths], sb[kFoldMaxWidths];
#pragma unroll
  for (int i = 0; i < kFoldMaxWidths; ++i) sw[i] = sb[i] = 0.0;
  for (int k = lane; k < D; k += 64) {
    const float wv = bf16_to_f32(w[k]);
    const uint16_t f = f32_to_bf16(gamma[k] * wv);
    wf[k] = f;
    const double fv = (double)bf16_to_f32(f), bv = (double)beta[k] * (double)wv;
#pragma unroll
    for (int i = 0; i < kFoldMaxWidths; ++i)
      if (i < wd.n && k < wd.e[i]) {
        sw[i] += fv;
        sb[i] += bv;
      }
  }
#pragma unroll
  for (int i = 0; i < kFoldMaxWidths; ++i) {
    if (i >= wd.n) break;
    double a = sw[i], c = sb[i];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      a += __shfl_xor(a, off, 64);
      c += __shfl_xor(c, off, 64);
    }
    if (lane == 0) {
      colsum[i * ldv + n] = (float)a;
      cbias[i * ldv + n] = (float)((double)bias[n] + c);
    }
  }
}

}  // namespace

hipError_t launch_layernorm_bf16(const void* x, int64_t x_stride, const float* xcls, int tokens,
                                 void* out, int64_t rows, int d, const float* g, const float* b,
                                 float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (xcls != nullptr && tokens < 1) return hipErrorInvalidValue;
  if ((d & 7) != 0 || d > 8 * 32 * kMaxChunks) return hipErrorInvalidValue;
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  uint16_t* op = static_cast<uint16_t*>(out);
  switch ((d + 255) / 256) {
    case 1: return launch_ln<1>(xp, x_stride, xcls, tokens, op, rows, d, g, b, eps, s);
    case 2: return launch_ln<2>(xp, x_stride, xcls, tokens, op, rows, d, g, b, eps, s);
    case 3: return launch_ln<3>(xp, x_stride, xcls, tokens, op, rows, d, g, b, eps, s);
    case 4: return launch_ln<4>(xp, x_stride, xcls, tokens, op, rows, d, g, b, eps, s);
    default: return launch_ln<kMaxChunks>(xp, x_stride, xcls, tokens, op, rows, d, g, b, eps, s);
  }
}

hipError_t launch_layernorm_f32(const void* x, int64_t x_stride, void* out, int64_t rows, int d,
                                const float* g, const float* b, float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int64_t blocks = (rows + 3) / 4;
  hipLaunchKernelGGL(layernorm_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     static_cast<const float*>(x), x_stride, static_cast<float*>(out), rows, d,
                     g, b, eps);
  return hipGetLastError();
}

hipError_t launch_ln_fold(const void* W, int N, int D, const float* gamma, const float* beta,
                          const float* bias, const int32_t* widths, int nw, void* Wf,
                          float* colsum, float* cbias, int64_t ldv, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (nw < 1 || nw > kFoldMaxWidths || D < 1 || ldv < N) return hipErrorInvalidValue;
  FoldWidths wd{};
  wd.n = nw;
  for (int i = 0; i < nw; ++i) {
    if (widths[i] < 1 || widths[i] > D) return hipErrorInvalidValue;
    wd.e[i] = widths[i];
  }
  hipLaunchKernelGGL(ln_fold_kernel, dim3((unsigned)((N + 3) / 4)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(W), N, D, gamma, beta, bias, wd,
                     static_cast<uint16_t*>(Wf), colsum, cbias, ldv);
  return hipGetLastError();
}

}  // namespace elasto
