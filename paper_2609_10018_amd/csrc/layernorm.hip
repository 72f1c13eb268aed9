// LayerNorm over the feature axis: u = (x - mean) / sqrt(var + eps) * g + b,
// biased variance, statistics in fp32.  Memory-bound: one wave per row, each
// lane holding its share of the row in registers (two passes over registers,
// one read of the row from HBM, one write).
//
// The bf16 path reads and writes 8-byte (4-element) bf16 vectors, so a wave
// moves 512 contiguous bytes per instruction; the class-token rows of the
// residual stream are fp32 and come from their own buffer.  Row stride is
// free.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

constexpr int kMaxVecPerLane = 8;  // 4-element vectors per lane: d <= 2048

__global__ __launch_bounds__(256) void layernorm_bf16_kernel(const uint16_t* __restrict__ x,
                                                             int64_t x_stride,
                                                             const float* __restrict__ xcls,
                                                             int tokens,
                                                             uint16_t* __restrict__ out,
                                                             int64_t rows, int d,
                                                             const float* __restrict__ g,
                                                             const float* __restrict__ b,
                                                             float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int nvec = d >> 2;
  const int64_t bi = xcls != nullptr ? row / tokens : 0;
  const bool cls_row = xcls != nullptr && row == bi * tokens;  // uniform per wave
  const uint16_t* xr = x + row * x_stride;
  const float* xc = cls_row ? xcls + bi * (int64_t)d : nullptr;
  float v[kMaxVecPerLane][4];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxVecPerLane; ++i) {
    const int vi = lane + 64 * i;
    if (vi < nvec) {
      if (cls_row) {
        const f32x4 w = *reinterpret_cast<const f32x4*>(xc + 4 * vi);
        v[i][0] = w[0];
        v[i][1] = w[1];
        v[i][2] = w[2];
        v[i][3] = w[3];
      } else {
        const u32x2 w = *reinterpret_cast<const u32x2*>(xr + 4 * vi);
        v[i][0] = __uint_as_float(w[0] << 16);
        v[i][1] = __uint_as_float(w[0] & 0xffff0000u);
        v[i][2] = __uint_as_float(w[1] << 16);
        v[i][3] = __uint_as_float(w[1] & 0xffff0000u);
      }
      s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
    } else {
      v[i][0] = v[i][1] = v[i][2] = v[i][3] = 0.0f;
    }
  }
  const float inv_d = 1.0f / (float)d;
  const float mean = wave_sum(s) * inv_d;
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxVecPerLane; ++i) {
    if (lane + 64 * i < nvec) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float c = v[i][e] - mean;
        ss += c * c;
      }
    }
  }
  const float rstd = rsqrtf(wave_sum(ss) * inv_d + eps);
  uint16_t* orow = out + row * (int64_t)d;
#pragma unroll
  for (int i = 0; i < kMaxVecPerLane; ++i) {
    const int vi = lane + 64 * i;
    if (vi < nvec) {
      const f32x4 gv = *reinterpret_cast<const f32x4*>(g + 4 * vi);
      const f32x4 bv = *reinterpret_cast<const f32x4*>(b + 4 * vi);
      uint16_t h[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = f32_to_bf16((v[i][e] - mean) * rstd * gv[e] + bv[e]);
      u32x2 w;
      w[0] = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
      w[1] = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
      *reinterpret_cast<u32x2*>(orow + 4 * vi) = w;
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

}  // namespace

hipError_t launch_layernorm_bf16(const void* x, int64_t x_stride, const float* xcls, int tokens,
                                 void* out, int64_t rows, int d, const float* g, const float* b,
                                 float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (xcls != nullptr && tokens < 1) return hipErrorInvalidValue;
  const int64_t blocks = (rows + 3) / 4;
  hipLaunchKernelGGL(layernorm_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     static_cast<const uint16_t*>(x), x_stride, xcls, tokens,
                     static_cast<uint16_t*>(out), rows, d, g, b, eps);
  return hipGetLastError();
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

}  // namespace elasto
