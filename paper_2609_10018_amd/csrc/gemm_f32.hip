// fp32 width-sliced GEMM, C[m][n] = epi(sum_k A[m][k] W[n][k] + bias[n]),
// on the vector ALU (fp32 FMA; no reduced-precision matrix mode).  A 64 x 64
// output tile per 256-thread workgroup, K staged 16 at a time in LDS, 4 x 4
// outputs per thread.  Any shape and stride: every load is bounds-checked and
// zero-filled, so nothing outside the active K prefix / N rows is read.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

struct P32 {
  const float* A;
  int64_t lda;
  const float* W;
  int64_t ldw;
  void* C;
  int64_t ldc;
  const float* bias;
  int64_t M;
  int N, K;
  const float* img;
  int img_size, patch, chans, grid, tokens;
  const float* cls;
  const float* pos;
  int64_t ldpos;
};

template <Epi E>
__global__ __launch_bounds__(256) void gemm_f32_kernel(P32 p) {
  __shared__ float As[16][64 + 4];
  __shared__ float Ws[16][64 + 4];
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)blockIdx.x * 64;
  const int n0 = blockIdx.y * 64;
  const int tx = tid & 15, ty = tid >> 4;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  for (int k0 = 0; k0 < p.K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + 256 * i, row = e >> 4, kk = e & 15;
      const int64_t gm = m0 + row;
      const int k = k0 + kk;
      float v = 0.f;
      if (gm < p.M && k < p.K) {
        if constexpr (E == Epi::Patch) {
          const int64_t bi = gm / p.tokens;
          const int t = (int)(gm - bi * p.tokens);
          if (t > 0) {
            const int n = t - 1, py = n / p.grid, px = n - py * p.grid;
            const int pp = p.patch * p.patch, c = k / pp, rem = k - c * pp;
            const int ii = rem / p.patch, jj = rem - ii * p.patch;
            v = p.img[((bi * p.chans + c) * p.img_size + py * p.patch + ii) * (int64_t)p.img_size +
                      px * p.patch + jj];
          }
        } else {
          v = p.A[gm * p.lda + k];
        }
      }
      As[kk][row] = v;
      const int gn = n0 + row;
      Ws[kk][row] = (gn < p.N && k < p.K) ? p.W[(int64_t)gn * p.ldw + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = Ws[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t row = m0 + ty * 4 + i;
    if (row >= p.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col >= p.N) continue;
      const float v = acc[i][j];
      const float bv = p.bias[col];
      float* c = static_cast<float*>(p.C) + row * p.ldc + col;
      if constexpr (E == Epi::Bias || E == Epi::BiasF32) {
        *c = v + bv;
      } else if constexpr (E == Epi::BiasGelu) {
        *c = gelu_erf(v + bv);
      } else if constexpr (E == Epi::BiasResid) {
        *c = *c + (v + bv);
      } else {
        const int t = (int)(row % p.tokens);
        *c = v + (t == 0 ? p.cls[col] : bv) + p.pos[(int64_t)t * p.ldpos + col];
      }
    }
  }
}

template <Epi E>
hipError_t launch(const P32& p, hipStream_t s) {
  const dim3 grid((unsigned)((p.M + 63) / 64), (unsigned)((p.N + 63) / 64));
  hipLaunchKernelGGL((gemm_f32_kernel<E>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_f32(Epi epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  P32 p{};
  p.A = static_cast<const float*>(a.A);
  p.lda = a.lda;
  p.W = static_cast<const float*>(a.W);
  p.ldw = a.ldw;
  p.C = a.C;
  p.ldc = a.ldc;
  p.bias = a.bias;
  p.M = a.M;
  p.N = a.N;
  p.K = a.K;
  p.img = static_cast<const float*>(a.img);
  p.img_size = a.img_size;
  p.patch = a.patch;
  p.chans = a.chans;
  p.grid = a.grid;
  p.tokens = a.tokens;
  p.cls = a.cls;
  p.pos = a.pos;
  p.ldpos = a.ldpos > 0 ? a.ldpos : a.N;
  switch (epi) {
    case Epi::Bias: return launch<Epi::Bias>(p, s);
    case Epi::BiasGelu: return launch<Epi::BiasGelu>(p, s);
    case Epi::BiasResid: return launch<Epi::BiasResid>(p, s);
    case Epi::BiasF32: return launch<Epi::BiasF32>(p, s);
    case Epi::Patch: return launch<Epi::Patch>(p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace elasto
