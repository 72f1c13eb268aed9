// Data-movement kernels of the elastic bottleneck-ResNet path (Section 4.1's
// CNN backbone, Table 2); the convolutions themselves run as bf16 MFMA GEMMs
// (gemm_bf16.hip, implicit for the 3x3 and strided 1x1 ones).  Activations
// are NHWC bf16.
//
// * pad_nhwc4: NCHW images (at most 4 channels) -> NHWC with 4 channels and
//   a zero border, the stem convolution's input: with 4 channels a 7-pixel
//   row of the stem's window is 56 contiguous bytes, read as one 64-byte run.
// * max_pool_3x3_s2: 3x3 window, stride 2, padding 1, NHWC, 8 channels per
//   thread.
// * avg_pool: mean over all pixels of each image, fp32 sums, bf16 out.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

inline unsigned grid_for(int64_t n, int block) { return (unsigned)((n + block - 1) / block); }

// One thread per padded output pixel: 4 channels (8 bytes), zero in the
// border and in channels >= C.
__global__ __launch_bounds__(256) void pad_nhwc4_kernel(const uint16_t* __restrict__ img, int C,
                                                        int H, int W, int pad, int64_t pixels,
                                                        uint16_t* __restrict__ out) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= pixels) return;
  const int Hp = H + 2 * pad, Wp = W + 2 * pad;
  const int64_t n = id / ((int64_t)Hp * Wp);
  const int r = (int)(id - n * Hp * Wp), y = r / Wp - pad, x = r - (r / Wp) * Wp - pad;
  uint32_t h[4] = {0u, 0u, 0u, 0u};
  if (y >= 0 && y < H && x >= 0 && x < W) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (c < C) h[c] = img[((n * C + c) * H + y) * (int64_t)W + x];
  }
  *reinterpret_cast<u32x2*>(out + id * 4) = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
}

__global__ __launch_bounds__(256) void max_pool_kernel(const uint16_t* __restrict__ x, int H, int W,
                                                       int C, int Ho, int Wo, int64_t outs,
                                                       uint16_t* __restrict__ y) {
  const int c8n = C / 8;
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= outs * c8n) return;
  const int64_t m = id / c8n;
  const int c8 = (int)(id - m * c8n);
  const int64_t n = m / ((int64_t)Ho * Wo);
  const int r = (int)(m - n * Ho * Wo), oh = r / Wo, ow = r - oh * Wo;
  float mx[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) mx[e] = -INFINITY;
#pragma unroll
  for (int i = 0; i < 3; ++i)
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const int ih = 2 * oh - 1 + i, iw = 2 * ow - 1 + j;
      if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
      const u32x4 v = *reinterpret_cast<const u32x4*>(x + ((n * H + ih) * W + iw) * (int64_t)C +
                                                      c8 * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        mx[e] = fmaxf(mx[e], __uint_as_float((e & 1) ? (v[e >> 1] & 0xffff0000u)
                                                      : (v[e >> 1] << 16)));
    }
  u32x4 w;
#pragma unroll
  for (int h = 0; h < 4; ++h)
    w[h] = (uint32_t)f32_to_bf16(mx[2 * h]) | ((uint32_t)f32_to_bf16(mx[2 * h + 1]) << 16);
  *reinterpret_cast<u32x4*>(y + m * (int64_t)C + c8 * 8) = w;
}

__global__ __launch_bounds__(256) void avg_pool_kernel(const uint16_t* __restrict__ x, int HW,
                                                       int C, int batch,
                                                       uint16_t* __restrict__ y) {
  const int c8n = C / 8;
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)batch * c8n) return;
  const int n = (int)(id / c8n), c8 = (int)(id - (int64_t)n * c8n);
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const uint16_t* p = x + (int64_t)n * HW * C + c8 * 8;
  for (int i = 0; i < HW; ++i) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p + (int64_t)i * C);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      s[e] += __uint_as_float((e & 1) ? (v[e >> 1] & 0xffff0000u) : (v[e >> 1] << 16));
  }
  const float inv = 1.0f / (float)HW;
  u32x4 w;
#pragma unroll
  for (int h = 0; h < 4; ++h)
    w[h] = (uint32_t)f32_to_bf16(s[2 * h] * inv) | ((uint32_t)f32_to_bf16(s[2 * h + 1] * inv) << 16);
  *reinterpret_cast<u32x4*>(y + (int64_t)n * C + c8 * 8) = w;
}

}  // namespace

hipError_t launch_pad_nhwc4(const void* img, int batch, int C, int H, int W, int pad, void* out,
                            hipStream_t s) {
  if (C < 1 || C > 4 || H < 1 || W < 1 || pad < 0) return hipErrorInvalidValue;
  const int64_t pixels = (int64_t)batch * (H + 2 * pad) * (W + 2 * pad);
  if (pixels <= 0) return hipSuccess;
  hipLaunchKernelGGL(pad_nhwc4_kernel, dim3(grid_for(pixels, 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(img), C, H, W, pad, pixels,
                     static_cast<uint16_t*>(out));
  return hipGetLastError();
}

hipError_t launch_max_pool_3x3_s2(const void* x, int batch, int H, int W, int C, void* y,
                                  hipStream_t s) {
  if ((C & 7) != 0) return hipErrorInvalidValue;
  const int Ho = (H - 1) / 2 + 1, Wo = (W - 1) / 2 + 1;
  const int64_t outs = (int64_t)batch * Ho * Wo, work = outs * (C / 8);
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(max_pool_kernel, dim3(grid_for(work, 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(x), H, W, C, Ho, Wo, outs,
                     static_cast<uint16_t*>(y));
  return hipGetLastError();
}

hipError_t launch_avg_pool(const void* x, int batch, int HW, int C, void* y, hipStream_t s) {
  if ((C & 7) != 0) return hipErrorInvalidValue;
  const int64_t work = (int64_t)batch * (C / 8);
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(avg_pool_kernel, dim3(grid_for(work, 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(x), HW, C, batch, static_cast<uint16_t*>(y));
  return hipGetLastError();
}

}  // namespace elasto
