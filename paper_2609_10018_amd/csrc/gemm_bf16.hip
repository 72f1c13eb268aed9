// Width-sliced bf16 GEMM on gfx950 matrix cores.
//
// C[m][n] = epi(sum_{k<K} A[m][k] * W[n][k] + bias[n]) with both operands
// K-contiguous ("NT").  Every linear layer of the elastic ViT is one of these:
// the mode only changes N (q/k/v rows of the active heads, fc1 rows of the
// active units: a contiguous prefix of the packed weight) or K (output
// projection and fc2 read a prefix of each packed weight row).
//
// Tiling: a 256-thread workgroup (4 waves, 2 x 2) owns a BM x BN output tile
// and walks K in steps of 64.  Each step's A and W tiles are staged in LDS
// (double-buffered, one barrier per step) with a 16-byte-chunk XOR swizzle so
// that the MFMA operand reads of 8 consecutive rows hit distinct banks.  Each
// wave computes a (BM/2) x (BN/2) block with v_mfma_f32_32x32x16_bf16
// (fp32 accumulate).  Ragged edges: rows past M / N re-read the last valid
// row (results discarded), K past the end is zero-filled element-wise in both
// operands, so inactive weights are never read into a product.
//
// Workgroups are renumbered so that each XCD (workgroup i runs on XCD i % 8)
// receives a contiguous run of row-major tiles: the tiles sharing an A panel
// then share that XCD's L2.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

constexpr int kBK = 64;
constexpr int kRowBytes = kBK * 2;

struct Params {
  const uint16_t* A;
  int64_t lda;
  const uint16_t* W;
  int64_t ldw;
  void* C;
  int64_t ldc;
  const float* bias;
  int M, N, K;
  const uint16_t* img;
  int img_size, patch, chans, grid, tokens;
  const float* cls;
  const float* pos;
  int tiles_n;
};

__device__ __forceinline__ int lds_off(int r, int c) {
  return r * kRowBytes + ((c ^ (r & 7)) << 4);
}

// Keep elements [kbeg, kend) of the 8-element chunk starting at kbeg.
__device__ __forceinline__ u32x4 mask_tail(u32x4 v, int kbeg, int kend) {
  u32x4 o;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int e = kbeg + 2 * w;
    const uint32_t lo = (e < kend) ? (v[w] & 0xffffu) : 0u;
    const uint32_t hi = (e + 1 < kend) ? (v[w] & 0xffff0000u) : 0u;
    o[w] = lo | hi;
  }
  return o;
}

template <int BM, int BN, Epi E>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(Params p) {
  constexpr int WM = 2, WN = 2;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int ACH = BM * 8 / 256, BCH = BN * 8 / 256;
  constexpr int STAGE = (BM + BN) * kRowBytes;
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  const int nblk = gridDim.x, b = blockIdx.x;
  const int q = nblk >> 3, r = nblk & 7, xcd = b & 7, idx = b >> 3;
  const int logical = (xcd < r) ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
  const int tile_m = logical / p.tiles_n, tile_n = logical - tile_m * p.tiles_n;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  const int cc = tid & 7;  // this thread's 16-byte chunk within a 128-byte row
  const uint16_t* asrc[ACH];
  bool azero[ACH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int gm = min(m0 + (tid >> 3) + 32 * i, p.M - 1);
    if constexpr (E == Epi::Patch) {
      const int bi = gm / p.tokens, t = gm - bi * p.tokens;
      const int n = t > 0 ? t - 1 : 0, py = n / p.grid, px = n - py * p.grid;
      azero[i] = (t == 0);
      asrc[i] = p.img + ((int64_t)bi * p.chans * p.img_size + (int64_t)py * p.patch) * p.img_size +
                px * p.patch;
    } else {
      azero[i] = false;
      asrc[i] = p.A + (int64_t)gm * p.lda;
    }
  }
  const uint16_t* bsrc[BCH];
#pragma unroll
  for (int j = 0; j < BCH; ++j) {
    const int gn = min(n0 + (tid >> 3) + 32 * j, p.N - 1);
    bsrc[j] = p.W + (int64_t)gn * p.ldw;
  }

  u32x4 ra[ACH], rb[BCH];
  auto load = [&](int k0) {
    const int k = k0 + cc * 8;
    const bool in = k < p.K, tail = k + 8 > p.K;
    int64_t aoff = k;
    if constexpr (E == Epi::Patch) {
      const int pp = p.patch * p.patch;
      const int c = k / pp, rem = k - c * pp, ii = rem / p.patch, jj = rem - ii * p.patch;
      aoff = ((int64_t)c * p.img_size + ii) * p.img_size + jj;
    }
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (in && !azero[i]) {
        v = *reinterpret_cast<const u32x4*>(asrc[i] + aoff);
        if (tail) v = mask_tail(v, k, p.K);
      }
      ra[i] = v;
    }
#pragma unroll
    for (int j = 0; j < BCH; ++j) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (in) {
        v = *reinterpret_cast<const u32x4*>(bsrc[j] + k);
        if (tail) v = mask_tail(v, k, p.K);
      }
      rb[j] = v;
    }
  };
  auto store = [&](char* stage) {
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      *reinterpret_cast<u32x4*>(stage + lds_off((tid >> 3) + 32 * i, cc)) = ra[i];
    char* bst = stage + BM * kRowBytes;
#pragma unroll
    for (int j = 0; j < BCH; ++j)
      *reinterpret_cast<u32x4*>(bst + lds_off((tid >> 3) + 32 * j, cc)) = rb[j];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  const int nk = (p.K + kBK - 1) / kBK;
  load(0);
  store(smem);
  __syncthreads();
  const int lr = lane & 31, lg = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const char* cur = smem + (kt & 1) * STAGE;
    if (kt + 1 < nk) load((kt + 1) * kBK);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int c = kk * 2 + lg;
      bf16x8 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(cur + lds_off(wm * WTM + i * 32 + lr, c));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bf[j] = *reinterpret_cast<const bf16x8*>(cur + BM * kRowBytes +
                                                 lds_off(wn * WTN + j * 32 + lr, c));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store(smem + ((kt + 1) & 1) * STAGE);
    __syncthreads();
  }

  // D layout of the 32x32 block: element e of lane l is
  // row 8*(e/4) + 4*(l/32) + e%4, column l%32.
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * WTN + j * 32 + lr;
      if (col >= p.N) continue;
      const float bv = p.bias[col];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + wm * WTM + i * 32 + 8 * (e >> 2) + 4 * lg + (e & 3);
        if (row >= p.M) continue;
        float v = acc[i][j][e];
        const int64_t o = (int64_t)row * p.ldc + col;
        if constexpr (E == Epi::Bias) {
          static_cast<uint16_t*>(p.C)[o] = f32_to_bf16(v + bv);
        } else if constexpr (E == Epi::BiasGelu) {
          static_cast<uint16_t*>(p.C)[o] = f32_to_bf16(gelu_erf(v + bv));
        } else if constexpr (E == Epi::BiasResid) {
          uint16_t* cp = static_cast<uint16_t*>(p.C);
          cp[o] = f32_to_bf16(bf16_to_f32(cp[o]) + (v + bv));
        } else if constexpr (E == Epi::BiasF32) {
          static_cast<float*>(p.C)[o] = v + bv;
        } else {  // Patch
          const int t = row % p.tokens;
          const float add = (t == 0 ? p.cls[col] : bv) + p.pos[(int64_t)t * p.N + col];
          static_cast<uint16_t*>(p.C)[o] = f32_to_bf16(v + add);
        }
      }
    }
  }
}

template <int BM, int BN, Epi E>
hipError_t launch_cfg(const Params& p0, hipStream_t s) {
  Params p = p0;
  const int64_t tm = (p.M + BM - 1) / BM, tn = (p.N + BN - 1) / BN;
  p.tiles_n = (int)tn;
  const int64_t blocks = tm * tn;
  if (blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, E>), dim3((unsigned)blocks), dim3(256), 0, s, p);
  return hipGetLastError();
}

template <Epi E>
hipError_t launch_epi(const Params& p, hipStream_t s) {
  // Pick the tile that keeps the chip busiest: estimated time is the number
  // of rounds of concurrent workgroups times the relative cost of one tile.
  struct Cfg { int bm, bn, per_cu; double rel; };
  const Cfg cfgs[3] = {{256, 256, 1, 1.0}, {256, 128, 1, 0.55}, {128, 128, 2, 0.30}};
  const int cus = 256;
  int best = 0;
  double best_t = 1e300;
  for (int i = 0; i < 3; ++i) {
    const int64_t tiles = ((p.M + cfgs[i].bm - 1) / cfgs[i].bm) * ((p.N + cfgs[i].bn - 1) / cfgs[i].bn);
    const int64_t slots = (int64_t)cus * cfgs[i].per_cu;
    const double t = (double)((tiles + slots - 1) / slots) * cfgs[i].rel * cfgs[i].per_cu;
    if (t < best_t - 1e-9) { best_t = t; best = i; }
  }
  switch (best) {
    case 0: return launch_cfg<256, 256, E>(p, s);
    case 1: return launch_cfg<256, 128, E>(p, s);
    default: return launch_cfg<128, 128, E>(p, s);
  }
}

}  // namespace

hipError_t launch_gemm_bf16(Epi epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  Params p{};
  p.A = static_cast<const uint16_t*>(a.A);
  p.lda = a.lda;
  p.W = static_cast<const uint16_t*>(a.W);
  p.ldw = a.ldw;
  p.C = a.C;
  p.ldc = a.ldc;
  p.bias = a.bias;
  p.M = (int)a.M;
  p.N = a.N;
  p.K = a.K;
  p.img = static_cast<const uint16_t*>(a.img);
  p.img_size = a.img_size;
  p.patch = a.patch;
  p.chans = a.chans;
  p.grid = a.grid;
  p.tokens = a.tokens;
  p.cls = a.cls;
  p.pos = a.pos;
  switch (epi) {
    case Epi::Bias: return launch_epi<Epi::Bias>(p, s);
    case Epi::BiasGelu: return launch_epi<Epi::BiasGelu>(p, s);
    case Epi::BiasResid: return launch_epi<Epi::BiasResid>(p, s);
    case Epi::BiasF32: return launch_epi<Epi::BiasF32>(p, s);
    case Epi::Patch: return launch_epi<Epi::Patch>(p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace elasto
