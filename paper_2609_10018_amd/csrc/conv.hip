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
// * stem_pool: the stem (7x7 stride-2 convolution + bias + ReLU) and the 3x3
//   stride-2 max pool in one kernel, reading the NCHW images directly: a
//   workgroup stages the input patch of an 8x8 block of pooled outputs
//   (39x40 pixels, 4 channels) and the filters in LDS, computes the 17x17
//   stem outputs the block's pooling windows cover with MFMAs, rounds them to
//   bf16 as the separate stem would store them, and pools them in LDS.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

typedef int16_t i16x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

// Two bf16 values packed in a 32-bit word.  Per 16-bit half: max with 0 as a
// signed integer (zero for a set sign bit), and max as an unsigned integer
// (the float max for non-negative values).
__device__ __forceinline__ uint32_t pk_relu_bf16(uint32_t a) {
  return __builtin_bit_cast(uint32_t,
                            __builtin_elementwise_max(__builtin_bit_cast(i16x2, a), (i16x2){0, 0}));
}
__device__ __forceinline__ uint32_t pk_max_u16(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, a),
                                                                __builtin_bit_cast(u16x2, b)));
}

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
    w[h] = pack_bf16x2(mx[2 * h], mx[2 * h + 1]);
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
    w[h] = pack_bf16x2(s[2 * h] * inv, s[2 * h + 1] * inv);
  *reinterpret_cast<u32x4*>(y + (int64_t)n * C + c8 * 8) = w;
}

// Fused stem + max pool (see the file comment).  One workgroup of 10 waves
// per (image, 8x8 block of pooled outputs).  Stem output (sh, sw) is
// relu(bias + sum over kernel row i, column j < 7, channel c < 4 of
// x[c][2sh - 3 + i][2sw - 3 + j] * w[n][i*32 + j*4 + c]) with x zero outside
// the image (and for c >= C); the packed filter row's 8th column and 4th
// channel hold zeros.  Pooled output (ph, pw) is the max of the stem outputs
// (2ph - 1 + di, 2pw - 1 + dj), di, dj < 3, inside the stem output.
constexpr int kStemPT = 8;                  // pooled outputs per block side
constexpr int kStemSR = 2 * kStemPT + 1;    // stem outputs per block side (17)
constexpr int kStemM = kStemSR * kStemSR;   // 289 stem outputs
constexpr int kStemMB = (kStemM + 31) / 32; // 10 row blocks of 32 (one per wave)
constexpr int kStemIR = 2 * kStemSR + 5;    // 39 input rows
constexpr int kStemIC = 2 * kStemSR + 6;    // 40 input columns (incl. the 8th tap column)
constexpr int kStemK = 7 * 32;              // 224 filter entries
constexpr int kStemWS = kStemK * 2 + 16;    // LDS row stride of a staged filter (bytes)
constexpr int kStemThreads = 64 * kStemMB;

// Byte offset of stem output m, channel n in the block's LDS copy: rows of N
// bf16, their 16-byte units permuted by (m mod 8) so that the 32 rows a
// wave's epilogue writes at once spread over the banks.
template <int N>
__device__ __forceinline__ int stem_slot(int m, int n) {
  return m * (N * 2) + ((((n >> 3) ^ m) & (N / 8 - 1)) << 4) + (n & 7) * 2;
}

template <int N>
__global__ __launch_bounds__(kStemThreads) void stem_pool_kernel(
    const uint16_t* __restrict__ img, int C, int S, const uint16_t* __restrict__ w, int ldw,
    const float* __restrict__ bias, uint16_t* __restrict__ out) {
  static_assert(N % 32 == 0 && N <= 64, "stem channels");
  constexpr int IN_BYTES = kStemIR * kStemIC * 8;
  constexpr int W_OFF = (IN_BYTES + 255) / 256 * 256;
  constexpr int GEMM_BYTES = W_OFF + N * kStemWS;
  constexpr int POOL_BYTES = kStemM * N * 2;
  __shared__ __attribute__((aligned(16))) char smem[GEMM_BYTES > POOL_BYTES ? GEMM_BYTES : POOL_BYTES];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int S2 = S / 2, S4 = S / 4, tiles = S4 / kStemPT;
  const int b = blockIdx.x / (tiles * tiles), t = blockIdx.x - b * tiles * tiles;
  const int ph0 = (t / tiles) * kStemPT, pw0 = (t - (t / tiles) * tiles) * kStemPT;
  const int y0 = 4 * ph0 - 5, x0 = 4 * pw0 - 5;  // image coordinates of the patch origin

  // Filters: N rows of 28 16-byte chunks.
  for (int q = tid; q < N * (kStemK / 8); q += kStemThreads) {
    const int n = q / (kStemK / 8), kc = q - n * (kStemK / 8);
    *reinterpret_cast<u32x4*>(smem + W_OFF + n * kStemWS + kc * 16) =
        *reinterpret_cast<const u32x4*>(w + (int64_t)n * ldw + kc * 8);
  }
  // Input patch, NHWC with 4 channels, zero outside the image: every load of
  // the thread's pixels is issued before the first LDS store.
  {
    constexpr int kIn = kStemIR * kStemIC, kSlots = (kIn + kStemThreads - 1) / kStemThreads;
    const uint16_t* const ib = img + (int64_t)b * C * S * S;
    uint32_t h[kSlots][4];
#pragma unroll
    for (int sl = 0; sl < kSlots; ++sl) {
      const int q = tid + sl * kStemThreads;
      const int lr = q / kStemIC, lc = q - lr * kStemIC, y = y0 + lr, x = x0 + lc;
      const bool ok = q < kIn && (unsigned)y < (unsigned)S && (unsigned)x < (unsigned)S;
      const uint32_t off = (uint32_t)(y * S + x) * 2u;  // bytes within a channel plane
#pragma unroll
      for (int c = 0; c < 4; ++c)
        h[sl][c] = (ok && c < C) ? (uint32_t)*reinterpret_cast<const uint16_t*>(
                                       reinterpret_cast<const char*>(ib + (int64_t)c * S * S) + off)
                                 : 0u;
    }
#pragma unroll
    for (int sl = 0; sl < kSlots; ++sl) {
      const int q = tid + sl * kStemThreads;
      if (q < kIn)
        *reinterpret_cast<u32x2*>(smem + q * 8) =
            u32x2{h[sl][0] | (h[sl][1] << 16), h[sl][2] | (h[sl][3] << 16)};
    }
  }
  __syncthreads();

  // D^T = W A^T per 32x32 block: wave = row block of stem outputs; lane l
  // holds stem output m = 32 wave + l % 32 and channels 8(e/4) + 4(l/32) + e%4.
  const int lr = lane & 31, lg = lane >> 5;
  const int m = min(wave * 32 + lr, kStemM - 1);
  const int r = m / kStemSR, c = m - r * kStemSR;
  f32x16 acc[N / 32];
#pragma unroll
  for (int nb = 0; nb < N / 32; ++nb)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[nb][e] = 0.0f;
#pragma unroll
  for (int kb = 0; kb < kStemK / 16; ++kb) {
    const int k8 = kb * 16 + lg * 8, i = k8 >> 5, q = (k8 & 31) >> 3;
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(smem + ((2 * r + i) * kStemIC + 2 * c + 2 * q) * 8);
#pragma unroll
    for (int nb = 0; nb < N / 32; ++nb) {
      const bf16x8 wf = *reinterpret_cast<const bf16x8*>(smem + W_OFF + (nb * 32 + lr) * kStemWS + k8 * 2);
      acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, a, acc[nb], 0, 0, 0);
    }
  }
  __syncthreads();  // every wave is done with the staged patch and filters

  // bias, rounded to bf16, then ReLU on the bf16 bits (a negative value's
  // sign bit makes it negative as a 16-bit integer; the same result as
  // rounding max(v, 0) for every finite v); stem outputs outside the image
  // hold 0 (a pooling window always has an output inside, and every output
  // is >= 0).
  const int mo = wave * 32 + lr;
  const int sh = 2 * ph0 - 1 + r, sw = 2 * pw0 - 1 + c;
  const bool inside = (unsigned)sh < (unsigned)S2 && (unsigned)sw < (unsigned)S2;
  if (mo < kStemM) {
#pragma unroll
    for (int nb = 0; nb < N / 32; ++nb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n0 = nb * 32 + 8 * g + 4 * lg;
        const f32x4 bz = *reinterpret_cast<const f32x4*>(bias + n0);
        uint32_t h[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const uint32_t v =
              pack_bf16x2(acc[nb][4 * g + 2 * e] + bz[2 * e], acc[nb][4 * g + 2 * e + 1] + bz[2 * e + 1]);
          h[e] = inside ? pk_relu_bf16(v) : 0u;
        }
        *reinterpret_cast<u32x2*>(smem + stem_slot<N>(mo, n0)) = u32x2{h[0], h[1]};
      }
  }
  __syncthreads();

  // Pool: one thread per (pooled output, 8 channels).  The stem outputs are
  // non-negative bf16, ordered as 16-bit unsigned integers.
  constexpr int C8 = N / 8;
  if (tid < kStemPT * kStemPT * C8) {
    const int pix = tid / C8, c8 = tid - pix * C8;
    const int pr = pix / kStemPT, pc = pix - pr * kStemPT;
    u32x4 o = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int di = 0; di < 3; ++di)
#pragma unroll
      for (int dj = 0; dj < 3; ++dj) {
        const int sm = (2 * pr + di) * kStemSR + 2 * pc + dj;
        const u32x4 v = *reinterpret_cast<const u32x4*>(smem + stem_slot<N>(sm, c8 * 8));
#pragma unroll
        for (int h = 0; h < 4; ++h) o[h] = pk_max_u16(o[h], v[h]);
      }
    const int ph = ph0 + pr, pw = pw0 + pc;
    *reinterpret_cast<u32x4*>(out + ((((int64_t)b * S4 + ph) * S4 + pw) * N + c8 * 8)) = o;
  }
}

}  // namespace

hipError_t launch_stem_pool(const void* img, int batch, int C, int S, const void* w, int ldw,
                            const float* bias, int N, void* out, hipStream_t s) {
  if (C < 1 || C > 4 || S < 32 || S % 32 != 0 || (N != 32 && N != 64) || ldw < kStemK ||
      ldw % 8 != 0 || reinterpret_cast<uintptr_t>(bias) % 16 != 0)
    return hipErrorInvalidValue;
  if (batch <= 0) return hipSuccess;
  const int tiles = S / 4 / kStemPT;
  const int64_t blocks = (int64_t)batch * tiles * tiles;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  if (N == 64)
    hipLaunchKernelGGL(stem_pool_kernel<64>, dim3((unsigned)blocks), dim3(kStemThreads), 0, s,
                       static_cast<const uint16_t*>(img), C, S, static_cast<const uint16_t*>(w),
                       ldw, bias, static_cast<uint16_t*>(out));
  else
    hipLaunchKernelGGL(stem_pool_kernel<32>, dim3((unsigned)blocks), dim3(kStemThreads), 0, s,
                       static_cast<const uint16_t*>(img), C, S, static_cast<const uint16_t*>(w),
                       ldw, bias, static_cast<uint16_t*>(out));
  return hipGetLastError();
}

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
