// Width-sliced bf16 GEMM on gfx950 matrix cores.
//
// C[m][n] = epi(sum_{k<K} A[m][k] * W[n][k] + bias[n]) with both operands
// K-contiguous ("NT").  Every linear layer of the elastic ViT is one of these:
// the mode only changes N (q/k/v rows of the active heads, fc1 rows of the
// active units: a contiguous prefix of the packed weight) or K (output
// projection and fc2 read a prefix of each packed weight row).
//
// Tiling: a workgroup owns a BM x BN output tile and walks K in steps of 64.
// Each step's A and W tiles land in LDS through direct global->LDS loads
// (global_load_lds_dwordx4: no staging registers), double-buffered, so the
// loads of step k+1 fly while step k is multiplied; one barrier per step.
// A 1-KB LDS block holds 8 rows x 128 B; the 16-byte chunks of a row are
// XOR-swizzled (chunk c of row r sits at c ^ ((r ^ r>>3) & 7)) so that the
// MFMA operand reads of 8 or 16 consecutive rows hit distinct banks.  The
// direct load writes lane l's 16 bytes at block + 16*l, so each lane fetches
// the global chunk that the swizzle maps to its slot.  Each wave multiplies a
// (BM/WM) x (BN/WN) block with v_mfma_f32_32x32x16_bf16 (fp32 accumulate).
//
// Ragged edges: rows past M / N re-read the last valid row (their results
// are discarded); when K is not a multiple of 64, the last K-step goes
// through registers instead, with every element at or past K zeroed in both
// operands, so inactive weights never enter a product.
//
// Implicit convolution (CONV kernels): A is an NHWC bf16 activation and
// output row m is pixel (image, oh, ow).  K walks the KH*KW taps, and within a
// tap the first Ca input channels: in steps of 64 when Ca > 32, otherwise
// 64 / Cp taps share one step (Cp = Ca rounded up to a power of two), so
// narrow modes do not multiply mostly zeros.  W row j keeps tap t's channels
// at j*ldw + t*wseg.  A and W land in LDS through range-checked buffer
// loads: a 16-byte chunk whose pixel lies in the zero padding, whose
// channels are at or past Ca, or whose tap is past the last, gets an offset
// past the end of the buffer and reads as zeros, so no patch matrix is ever
// written to memory.
//
// Workgroups are renumbered so that each XCD (workgroup i runs on XCD i % 8)
// receives a contiguous run of tiles, ordered in groups of row panels so that
// the tiles an XCD runs at the same time share A and W panels in its L2.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;

constexpr int kBK = 64;        // K per step
constexpr int kRowBytes = 128; // one LDS row: 64 bf16
constexpr int kRowsPerBlock = 8;

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
  int64_t ldpos;
  float* ccls;
  int row0;     // this launch covers rows [row0, M)
  int tiles_n;
  int group_m;  // row panels per rasterisation group
  int relu;     // Bias / BiasResid: clamp the bf16 result at 0 (convolution blocks)
  int plan;     // forced tile plan (GemmArgs::plan), 0: the planner
  // Implicit convolution: input [*, H, W, Cs] (first Ca channels active),
  // KH x KW taps (row-major), stride, zero padding, output Ho x Wo; weights
  // stride wseg elements per tap; nc = 64-channel steps per tap; buffer
  // sizes in bytes (each below 2^31) for the range checks.
  // tps = taps per K step (1: nc steps per tap; > 1: each tap spans 2^cshift
  // elements of the step); tap / KW = (tap * kwinv) >> 16.
  int cv_H, cv_W, cv_Cs, cv_Ca, cv_KW, cv_T, cv_stride, cv_pad, cv_Ho, cv_Wo, cv_wseg, cv_nc;
  int cv_tps, cv_cshift, cv_kwinv;
  int cv_ncinv;     // K step / nc = (step * cv_ncinv) >> 16 (exact for every step)
  int cv_rowb, cv_pixb;  // bytes of one input row (W * Cs * 2) and one pixel (Cs * 2)
  int patch_shift;  // Patch: log2(patch) when patch is a power of two, else -1
  int a_bytes, w_bytes;
  // BiasResid residual source (nullptr: C itself); BiasGelu pre-activation
  // output / GeluBwd pre-activation input (nullptr: none).
  const uint16_t* res;
  int64_t ldres;
  uint16_t* aux;
  int64_t ldaux;
  // BiasF32 split-K: blockIdx.y = chunk of kchunk K-elements, partial
  // product to C + chunk * c_split.
  int ksplit, kchunk;
  int64_t c_split;
  // LayerNorm folding (see GemmArgs): producer statistics out, consumer
  // statistics in, the consumer's column sums, epsilon.
  float2* ln_out;
  const float2* ln_in;
  int64_t ln_ld;
  const float* ln_colsum;
  float ln_eps;
};

// Lane exchanges within a DPP row: quad_perm (1,0,3,2) and (2,3,0,1) swap
// neighbours 1 and 2 apart; row_half_mirror maps lane i of each 8-lane half
// to 7 - i.  The three together reach every lane of an aligned group of 8.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141;

// LayerNorm statistics.  The GEMM that writes a row of the residual stream
// stores, for each of the row's 64-column segments j (n_j = min(64, K - 64 j)
// columns), the pair (S_j, M2_j): the sum of the segment's values and the sum
// of their squared deviations from the segment's mean.  Pairs are merged with
// the pairwise update of Chan, Golub and LeVeque: for counts n_a, n_b, means
// m_a, m_b and deviation sums M2_a, M2_b, with d = m_b - m_a and n = n_a + n_b,
//   mean = m_a + d n_b / n,   M2 = M2_a + M2_b + d^2 n_a n_b / n,
// which never subtracts two large sums, so rows whose mean is large against
// their spread keep an accurate variance.
struct LnStat {
  float n, mean, m2;
};

__device__ __forceinline__ void ln_merge(LnStat& a, float nb, float mb, float m2b) {
  const float n = a.n + nb;
  const float f = n > 0.0f ? nb * __builtin_amdgcn_rcpf(n) : 0.0f;
  const float d = mb - a.mean;
  a.mean = fmaf(d, f, a.mean);
  a.m2 += fmaf(d * d, a.n * f, m2b);
  a.n = n;
}

// Merge into `a` the statistics held by the lane selected by DPP control CTRL.
template <int CTRL>
__device__ __forceinline__ void ln_merge_dpp(LnStat& a) {
  const float nb = dpp_f<CTRL>(a.n), mb = dpp_f<CTRL>(a.mean), m2b = dpp_f<CTRL>(a.m2);
  ln_merge(a, nb, mb, m2b);
}

// The same update for two sets of equal size (n_b = n_a, a power of two):
// d n_b / n = d / 2 and n_a n_b / n = n_a / 2, with no reciprocal.
__device__ __forceinline__ void ln_merge_equal(LnStat& a, float mb, float m2b) {
  const float d = mb - a.mean;
  a.mean = fmaf(d, 0.5f, a.mean);
  a.m2 += fmaf(d * d, a.n * 0.5f, m2b);
  a.n += a.n;
}
template <int CTRL>
__device__ __forceinline__ void ln_merge_dpp_equal(LnStat& a) {
  ln_merge_equal(a, dpp_f<CTRL>(a.mean), dpp_f<CTRL>(a.m2));
}


// Statistics of 8 values (all of them valid, or none).
__device__ __forceinline__ LnStat ln_of8(const float* v, bool valid) {
  LnStat s{0.0f, 0.0f, 0.0f};
  if (valid) {
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) t += v[e];
    const float m = t * 0.125f;
    float q = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) q = fmaf(v[e] - m, v[e] - m, q);
    s = LnStat{8.0f, m, q};
  }
  return s;
}

// Segment statistics from the 8-value chunks held by the 8 lanes of an
// aligned group.  When N is a multiple of 64 the chunks of a segment inside
// [0, N) are all whole, so the three merges are of equal sizes.
__device__ __forceinline__ LnStat ln_of_group8(const float* v, bool valid, bool whole_segments) {
  LnStat ls = ln_of8(v, valid);
  if (whole_segments) {
    ln_merge_dpp_equal<kDppXor1>(ls);
    ln_merge_dpp_equal<kDppXor2>(ls);
    ln_merge_dpp_equal<kDppHalfMirror>(ls);
  } else {
    ln_merge_dpp<kDppXor1>(ls);
    ln_merge_dpp<kDppXor2>(ls);
    ln_merge_dpp<kDppHalfMirror>(ls);
  }
  return ls;
}

// Merges, in segment order, the segments of a row (stored row-major: segment j
// of row r at part[r * ld + j], ld even so that segments 2i and 2i+1 form one
// 16-byte load) whose pair index is i = first, first + step, ... <
// ceil(nseg / 2), four loads in flight at a time.  Branch-free: a pair past
// the last re-reads pair 0, and a segment past the last (n_j <= 0) merges as
// an empty one.
__device__ __forceinline__ void ln_sums(const float2* row, int K, int first, int step, LnStat& st) {
  const int nseg = (K + 63) >> 6, npair = (nseg + 1) >> 1;
  for (int i0 = first; i0 < npair; i0 += 4 * step) {
    f32x4 q[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int i = i0 + t * step;
      q[t] = *reinterpret_cast<const f32x4*>(row + 2 * (i < npair ? i : 0));
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int i = i0 + t * step;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int nj = i < npair ? min(64, K - 64 * (2 * i + h)) : 0;
        const float nb = (float)max(nj, 0);
        ln_merge(st, nb, q[t][2 * h] * __builtin_amdgcn_rcpf(fmaxf(nb, 1.0f)),
                 nj > 0 ? q[t][2 * h + 1] : 0.0f);
      }
    }
  }
}

// (rstd, -rstd * mean) of a row from its merged statistics (biased variance).
__device__ __forceinline__ float2 ln_factors(const LnStat& st, float eps) {
  const float var = fmaxf(st.m2 * __builtin_amdgcn_rcpf(st.n), 0.0f);
  const float rstd = 1.0f / sqrtf(var + eps);
  return make_float2(rstd, -rstd * st.mean);
}

// Buffer descriptor word 3 for raw (unswizzled, stride 0) buffers on CDNA.
constexpr int kRsrcWord3 = 0x00020000;
constexpr unsigned kOutOfRange = 0x80000000u;  // at or past every buffer's size

__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

// Wait until at most N vector-memory operations of this wave are in flight
// and every LDS operation has completed.
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

// Wait until every LDS operation of this wave has completed (vector memory
// operations may still be in flight).
__device__ __forceinline__ void wait_lds() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14));
}

// Store 8 floats (the first `valid` of them when the chunk is ragged).
__device__ __forceinline__ void store_f32x8(float* cp, const float* v, bool full, int valid) {
  if (full) {
    *reinterpret_cast<f32x4*>(cp) = f32x4{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(cp + 4) = f32x4{v[4], v[5], v[6], v[7]};
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (e < valid) cp[e] = v[e];
  }
}

// Store 8 values rounded to bf16 (the first `valid` of them when ragged).
__device__ __forceinline__ void store_bf16x8(uint16_t* cp, const float* v, bool full, int valid) {
  if (full) {
    u32x4 w;
#pragma unroll
    for (int h = 0; h < 4; ++h)
      w[h] = pack_bf16x2(v[2 * h], v[2 * h + 1]);
    *reinterpret_cast<u32x4*>(cp) = w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (e < valid) cp[e] = f32_to_bf16(v[e]);
  }
}

// Keep elements [kbeg, kend) of the 8-element chunk starting at kbeg.
__device__ __forceinline__ u32x4 mask_tail(u32x4 v, int kbeg, int kend) {
  u32x4 o;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int e = kbeg + 2 * w;
    const uint32_t lo = (e < kend) ? 0x0000ffffu : 0u;
    const uint32_t hi = (e + 1 < kend) ? 0xffff0000u : 0u;
    o[w] = v[w] & (lo | hi);
  }
  return o;
}

// STAGES: LDS stages of the tile loads (2: the next K step in flight while
// this one computes; 4: three steps in flight, for launches of few tiles whose
// K chain is bound by the load latency; needs K % 64 == 0 and no CONV).
template <int BM, int BN, int WM, int WN, Epi E, bool CONV, int STAGES = 2>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_kernel(Params p) {
  static_assert(STAGES == 2 || (STAGES == 4 && !CONV), "stage counts");
  constexpr int NW = WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int ABLK = BM / kRowsPerBlock, BBLK = BN / kRowsPerBlock;
  constexpr int PER_WAVE = (ABLK + BBLK) / NW;
  // Gathering loaders (convolutions, patches): load i of wave w brings block
  // i * NW + w, so loads i < APW are A blocks and the rest W blocks for every
  // wave, and whether a load gathers is known at compile time (no branch on
  // the wave index in the K loop).  Plain GEMMs keep contiguous blocks per
  // wave (block w * PER_WAVE + i), measured faster for them.
  constexpr bool GATHER = CONV || E == Epi::Patch;
  constexpr int APW = ABLK / NW;
  static_assert(ABLK % NW == 0 && BBLK % NW == 0, "blocks must split evenly over waves");
  constexpr int STAGE = (BM + BN) * kRowBytes;
  constexpr int EPI_BYTES = (BM > 128 ? 128 : BM) * (BN + 8) * 4;
  constexpr int SMEM_MAIN = STAGES * STAGE > EPI_BYTES ? STAGES * STAGE : EPI_BYTES;
  constexpr bool LN_CONSUMER = E == Epi::Bias || E == Epi::BiasGelu;
  constexpr bool LN_PRODUCER = E == Epi::BiasResid || E == Epi::Patch;
  constexpr int SMEM = SMEM_MAIN;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  // Per-row LayerNorm factors of a folded LayerNorm (BM float2): dynamic LDS
  // that the launch adds only when the GEMM consumes one, so plain GEMMs keep
  // their occupancy.
  extern __shared__ __attribute__((aligned(16))) char smem_ln[];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if constexpr (E == Epi::BiasF32) {
    if (p.ksplit > 1) {
      const int k0 = blockIdx.y * p.kchunk;
      p.A += k0;
      p.W += k0;
      p.K = min(p.kchunk, p.K - k0);
      p.C = static_cast<float*>(p.C) + blockIdx.y * p.c_split;
    }
  }
  const int wm = wave / WN, wn = wave % WN;

  // Tile order: workgroup i runs on XCD i % 8, so each XCD first receives a
  // contiguous run of logical tile ids; logical ids then walk groups of
  // group_m row panels, N tiles within a group, row panels innermost, so the
  // tiles an XCD runs together share few A and W panels in its L2.
  const int nblk = gridDim.x, b = blockIdx.x;
  const int q = nblk >> 3, r8 = nblk & 7, xcd = b & 7, idx = b >> 3;
  const int logical = (xcd < r8) ? xcd * (q + 1) + idx : r8 * (q + 1) + (xcd - r8) * q + idx;
  const int tiles_m = (p.M - p.row0 + BM - 1) / BM;
  const int group = logical / (p.group_m * p.tiles_n), in_group = logical - group * p.group_m * p.tiles_n;
  const int gm = min(p.group_m, tiles_m - group * p.group_m);
  const int tile_n = in_group / gm, tile_m = group * p.group_m + (in_group - tile_n * gm);
  const int m0 = p.row0 + tile_m * BM, n0 = tile_n * BN;

  // Per block this lane loads: the row start, the logical 16-byte chunk, and
  // the block's LDS offset within a stage.
  const uint16_t* src[PER_WAVE];
  int chunk[PER_WAVE];
  int ldsoff[PER_WAVE];
  // CONV: element offset of the row's tap-0 pixel (A) or of the weight row
  // (W), and (A) the taps that fall inside the image: bit t of tmask is set
  // when tap t (kernel row t / KW, column t % KW) of the row's output pixel
  // reads an input pixel, so a K step tests one bit instead of two ranges.
  int cbase[PER_WAVE];
  uint64_t tmask[PER_WAVE];
  // CONV with several taps per K step (cv_tps > 1): the lane's tap within a
  // step (dtap), and its byte offset without the tap term: A, the tap-0
  // pixel plus the channel; W, the weight row plus the tap's segment and the
  // channel.  A chunk past the active channels clears the row's tap mask
  // (A) or wok (W).
  int dtap[PER_WAVE], boff[PER_WAVE];
  bool wok[PER_WAVE];
  const int prow = lane >> 3, pc = lane & 7;
#pragma unroll
  for (int i = 0; i < PER_WAVE; ++i) {
    const int blk = GATHER ? i * NW + wave : wave * PER_WAVE + i;
    if (GATHER ? i < APW : blk < ABLK) {
      const int r = blk * kRowsPerBlock + prow;
      const int gm = min(m0 + r, p.M - 1);
      chunk[i] = pc ^ swz(r);
      ldsoff[i] = blk * 1024;
      if constexpr (CONV) {
        const int hw = p.cv_Ho * p.cv_Wo, im = gm / hw, rem = gm - im * hw;
        const int oh = rem / p.cv_Wo, ow = rem - oh * p.cv_Wo;
        const int ih = oh * p.cv_stride - p.cv_pad, iw = ow * p.cv_stride - p.cv_pad;
        cbase[i] = ((im * p.cv_H + ih) * p.cv_W + iw) * p.cv_Cs;
        // Keep the product itself in a register: folding the tap offset into
        // its factors would put a multiply into every load of the K loop.
        asm volatile("" : "+v"(cbase[i]));
        uint64_t m = 0;
        for (int t = 0; t < p.cv_T; ++t) {
          const int ti = (t * p.cv_kwinv) >> 16, tj = t - ti * p.cv_KW;
          const bool in = ((unsigned)(ih + ti) < (unsigned)p.cv_H) &
                          ((unsigned)(iw + tj) < (unsigned)p.cv_W);
          m |= (uint64_t)in << t;
        }
        tmask[i] = m;
        if (p.cv_tps > 1) {
          const int q = chunk[i] * 8, ch = q & ((1 << p.cv_cshift) - 1);
          dtap[i] = q >> p.cv_cshift;
          boff[i] = (cbase[i] + ch) * 2;
          if (ch >= p.cv_Ca) tmask[i] = 0;
          wok[i] = false;
        }
        src[i] = nullptr;
      } else if constexpr (E == Epi::Patch) {
        const int bi = gm / p.tokens, t = gm - bi * p.tokens;
        const int n = t > 0 ? t - 1 : 0, py = n / p.grid, px = n - py * p.grid;
        src[i] = p.img + ((int64_t)bi * p.chans * p.img_size + (int64_t)py * p.patch) * p.img_size +
                 px * p.patch;
      } else {
        src[i] = p.A + (int64_t)gm * p.lda;
      }
    } else {
      const int r = (blk - ABLK) * kRowsPerBlock + prow;
      chunk[i] = pc ^ swz(r);
      ldsoff[i] = BM * kRowBytes + (blk - ABLK) * 1024;
      src[i] = p.W + (int64_t)min(n0 + r, p.N - 1) * p.ldw;
      if constexpr (CONV) {
        cbase[i] = min(n0 + r, p.N - 1) * (int)p.ldw;
        tmask[i] = 0;
        if (p.cv_tps > 1) {
          const int q = chunk[i] * 8, ch = q & ((1 << p.cv_cshift) - 1);
          dtap[i] = q >> p.cv_cshift;
          boff[i] = (cbase[i] + dtap[i] * p.cv_wseg + ch) * 2;
          wok[i] = ch < p.cv_Ca;
        }
      }
    }
  }
  // Patch rows with a power-of-two patch of at least 8: a K step (64 values)
  // stays in one channel and covers whole patch rows, so the im2col offset
  // of (step kt, chunk q) splits into a per-step part, the same for every
  // lane, and a per-chunk part fixed for the row block (plofs).
  int plofs[PER_WAVE];
  if constexpr (E == Epi::Patch) {
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int q = chunk[i] * 8, sh = p.patch_shift > 0 ? p.patch_shift : 0;
      plofs[i] = (q >> sh) * p.img_size + (q & (p.patch - 1));
    }
  }
  const bool patch_fast = E == Epi::Patch && p.patch_shift >= 3;
  // Element offset of k-index k within a source row (im2col for patches).
  auto koff = [&](int i, int k) -> int64_t {
    if constexpr (E == Epi::Patch) {
      if (i < APW) {
        int c, ii, jj;
        if (p.patch_shift >= 0) {
          const int sh = p.patch_shift, msk = p.patch - 1;
          c = k >> (2 * sh);
          ii = (k >> sh) & msk;
          jj = k & msk;
        } else {
          const int pp = p.patch * p.patch;
          c = k / pp;
          const int rem = k - c * pp;
          ii = rem / p.patch;
          jj = rem - ii * p.patch;
        }
        return ((int64_t)c * p.img_size + ii) * p.img_size + jj;
      }
    }
    return k;
  };

  const int nk_full = !CONV ? p.K / kBK
                      : p.cv_tps == 1 ? p.cv_T * p.cv_nc
                                      : (p.cv_T + p.cv_tps - 1) / p.cv_tps;
  const int nk = CONV ? nk_full : (p.K + kBK - 1) / kBK;
  // Buffer descriptors of the CONV loads (unused otherwise).
  const __amdgpu_buffer_rsrc_t rs_a =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.A), (short)0, p.a_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rs_w =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.W), (short)0, p.w_bytes, kRsrcWord3);
  // Loads blocks [lo, hi) of K step kt into stage `stage`.
  auto issue = [&](int stage, int kt, int lo, int hi) {
    char* base = smem + stage * STAGE;
    if constexpr (CONV) {
      if (p.cv_tps > 1) {
        // Several taps per step: this lane's chunk belongs to tap t0 + dtap.
        // The host guarantees that every tap offset and every t * kwinv fit
        // 24 bits, so the tap's pixel offset takes 24-bit multiplies.
        const int t0 = kt * p.cv_tps;
#pragma unroll
        for (int i = 0; i < PER_WAVE; ++i) {
          if (i < lo || i >= hi) continue;
          const int t = t0 + dtap[i];
          if (i < APW) {
            const int ti = (int)(__umul24((unsigned)t, (unsigned)p.cv_kwinv) >> 16);
            const int tj = t - (int)__umul24((unsigned)ti, (unsigned)p.cv_KW);
            const int toff = (int)(__umul24((unsigned)ti, (unsigned)p.cv_rowb) +
                                   __umul24((unsigned)tj, (unsigned)p.cv_pixb));
            const bool ok = (t < p.cv_T) & (bool)((tmask[i] >> (t & 63)) & 1u);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_a, (lds_void*)(base + ldsoff[i]), 16,
                                                     ok ? (unsigned)(boff[i] + toff) : kOutOfRange,
                                                     0, 0, 0);
          } else {
            const bool ok = (t < p.cv_T) & wok[i];
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs_w, (lds_void*)(base + ldsoff[i]), 16,
                ok ? (unsigned)(boff[i] + t0 * p.cv_wseg * 2) : kOutOfRange, 0, 0, 0);
          }
        }
        return;
      }
      const int t = (kt * p.cv_ncinv) >> 16, c0 = (kt - t * p.cv_nc) * kBK;
      const int ti = (t * p.cv_kwinv) >> 16, tj = t - ti * p.cv_KW;
      const int tap = (ti * p.cv_W + tj) * p.cv_Cs, wtap = t * p.cv_wseg;
#pragma unroll
      for (int i = 0; i < PER_WAVE; ++i) {
        if (i < lo || i >= hi) continue;
        const int ch = c0 + chunk[i] * 8;
        if (i < APW) {
          const bool ok = (ch < p.cv_Ca) & (bool)((tmask[i] >> t) & 1u);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rs_a, (lds_void*)(base + ldsoff[i]), 16,
              ok ? (unsigned)(cbase[i] + tap + ch) * 2u : kOutOfRange, 0, 0, 0);
        } else {
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rs_w, (lds_void*)(base + ldsoff[i]), 16,
              ch < p.cv_Ca ? (unsigned)(cbase[i] + wtap + ch) * 2u : kOutOfRange, 0, 0, 0);
        }
      }
    } else if (kt < nk_full) {
      // Patch rows, fast form: offset of step kt's channel and patch row.
      int64_t patch_step = 0;
      if constexpr (E == Epi::Patch) {
        if (patch_fast) {
          const int k0 = kt * kBK, sh = p.patch_shift;
          patch_step = (int64_t)(k0 >> (2 * sh)) * p.img_size * p.img_size +
                       (int64_t)((k0 & (p.patch * p.patch - 1)) >> sh) * p.img_size;
        }
      }
#pragma unroll
      for (int i = 0; i < PER_WAVE; ++i)
        if (i >= lo && i < hi)
        __builtin_amdgcn_global_load_lds(
            (global_void*)(src[i] + ((E == Epi::Patch && i < APW && patch_fast)
                                         ? patch_step + plofs[i]
                                         : koff(i, kt * kBK + chunk[i] * 8))),
            (lds_void*)(base + ldsoff[i]), 16, 0, 0);
    } else {
      // Ragged last step: masked loads through registers.
      u32x4 v[PER_WAVE];
#pragma unroll
      for (int i = 0; i < PER_WAVE; ++i) {
        const int k = kt * kBK + chunk[i] * 8;
        const bool in = k < p.K;
        v[i] = *reinterpret_cast<const u32x4*>(src[i] + koff(i, in ? k : 0));
        v[i] = mask_tail(v[i], k, p.K);
      }
#pragma unroll
      for (int i = 0; i < PER_WAVE; ++i)
        *reinterpret_cast<u32x4*>(base + ldsoff[i] + lane * 16) = v[i];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  const int lr = lane & 31, lg = lane >> 5;
  if constexpr (STAGES == 2) issue(0, 0, 0, PER_WAVE);
  else {
#pragma unroll
    for (int s0 = 0; s0 < STAGES - 1; ++s0)
      if (s0 < nk) issue(s0, s0, 0, PER_WAVE);
  }
  for (int kt = 0; kt < nk; ++kt) {
    if constexpr (STAGES == 2) {
      wait_vm_lds<0>();
      __builtin_amdgcn_s_barrier();
      if (kt + 1 < nk) issue((kt + 1) & 1, kt + 1, 0, PER_WAVE);
    } else {
      // Step kt's loads have landed when no more than the later steps' loads
      // (PER_WAVE each, issued in order) are in flight.
      const int ahead = min(STAGES - 2, nk - 1 - kt);
      if (ahead >= 2) wait_vm_lds<2 * PER_WAVE>();
      else if (ahead == 1) wait_vm_lds<PER_WAVE>();
      else wait_vm_lds<0>();
      __builtin_amdgcn_s_barrier();
      // The stage of step kt - 1, which every wave has finished reading.
      if (kt + STAGES - 1 < nk) issue((kt + STAGES - 1) % STAGES, kt + STAGES - 1, 0, PER_WAVE);
    }
    const char* cur = smem + (STAGES == 2 ? (kt & 1) : (kt % STAGES)) * STAGE;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int c = kk * 2 + lg;
      bf16x8 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WTM + i * 32 + lr;
        af[i] = *reinterpret_cast<const bf16x8*>(cur + r * kRowBytes + ((c ^ swz(r)) << 4));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WTN + j * 32 + lr;
        bf[j] = *reinterpret_cast<const bf16x8*>(cur + BM * kRowBytes + r * kRowBytes +
                                                 ((c ^ swz(r)) << 4));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  }

  // Epilogue.  The fp32 tile goes through LDS (in passes of up to 128 rows)
  // so that bias, activation, residual and conversion run on 8-column chunks
  // with 16-byte global loads and stores.  D layout of a 32x32 MFMA block:
  // element e of lane l is row 8*(e/4) + 4*(l/32) + e%4, column l%32.
  constexpr int SR = BM > 128 ? 128 : BM;  // rows per pass
  constexpr int SS = BN + 8;                // staged row stride (floats): the two
                                            // half-waves land on distinct banks
  constexpr int CPR = BN / 8;               // 8-column chunks per row
  constexpr int NT = 64 * NW;
  constexpr int RSTEP = NT / CPR;           // rows between one thread's chunks
  constexpr int ITER = SR / RSTEP;          // chunks per thread per pass
  static_assert(NT % CPR == 0 && SR % RSTEP == 0, "epilogue chunking");
  float* stg = reinterpret_cast<float*>(smem);

  // A thread always handles the same 8 columns: load their bias once.
  const int cc = tid % CPR, r_first = tid / CPR;
  const int col = n0 + cc * 8;
  const bool col_in = col < p.N, full = col + 8 <= p.N;
  float bv[8];
  if (p.bias == nullptr || E == Epi::GeluBwd) {  // no bias term
#pragma unroll
    for (int e = 0; e < 8; ++e) bv[e] = 0.0f;
  } else if (full) {
    const f32x4 b0 = *reinterpret_cast<const f32x4*>(p.bias + col);
    const f32x4 b1 = *reinterpret_cast<const f32x4*>(p.bias + col + 4);
    bv[0] = b0[0]; bv[1] = b0[1]; bv[2] = b0[2]; bv[3] = b0[3];
    bv[4] = b1[0]; bv[5] = b1[1]; bv[6] = b1[2]; bv[7] = b1[3];
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) bv[e] = col + e < p.N ? p.bias[col + e] : 0.0f;
  }

  // Folded LayerNorm (consumer): column sums of this thread's 8 columns, and
  // (rstd, -rstd * mean) of the tile's rows into LDS.
  float cs[8];
  float2* rowst = reinterpret_cast<float2*>(smem_ln);
  if constexpr (LN_CONSUMER && !CONV) {
    if (p.ln_in != nullptr) {
#pragma unroll
      for (int e = 0; e < 8; ++e) cs[e] = col + e < p.N ? p.ln_colsum[col + e] : 0.0f;
      if (tid < BM) {
        LnStat st{0.0f, 0.0f, 0.0f};
        ln_sums(p.ln_in + (int64_t)min(m0 + tid, p.M - 1) * p.ln_ld, p.K, 0, 1, st);
        rowst[tid] = ln_factors(st, p.ln_eps);
      }
    }
  }

  wait_lds();  // every wave has finished reading the last stage
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int pass = 0; pass < BM / SR; ++pass) {
    const int row_base = m0 + pass * SR + r_first;
    // Residual rows of this pass: issued before the staging so that their
    // latency overlaps it.
    u32x4 res[ITER];
    if constexpr (E == Epi::BiasResid || E == Epi::GeluBwd) {
      const uint16_t* rsrc = E == Epi::GeluBwd ? p.aux
                             : p.res != nullptr ? p.res : static_cast<const uint16_t*>(p.C);
      const int64_t rld = E == Epi::GeluBwd ? p.ldaux : p.res != nullptr ? p.ldres : p.ldc;
#pragma unroll
      for (int it = 0; it < ITER; ++it) {
        const int row = row_base + it * RSTEP;
        res[it] = (full && row < p.M)
                      ? *reinterpret_cast<const u32x4*>(rsrc + (int64_t)row * rld + col)
                      : u32x4{0u, 0u, 0u, 0u};
      }
    }
    if ((wm * WTM) / SR == pass) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int rl = (wm * WTM) % SR + i * 32 + 8 * (e >> 2) + 4 * lg + (e & 3);
            stg[rl * SS + wn * WTN + j * 32 + lr] = acc[i][j][e];
          }
    }
    wait_lds();
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int rl = r_first + it * RSTEP;
      const int row = row_base + it * RSTEP;
      if (row >= p.M) continue;  // the same row for every lane of an 8-lane group
      // Values whose LayerNorm statistics this lane contributes (producers).
      float st[8];
      bool st_ok = false;
      if (col_in) do {
      const f32x4 s0 = *reinterpret_cast<const f32x4*>(stg + rl * SS + cc * 8);
      const f32x4 s1 = *reinterpret_cast<const f32x4*>(stg + rl * SS + cc * 8 + 4);
      float v[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
      const int64_t o = (int64_t)row * p.ldc + col;
      if constexpr (E == Epi::BiasF32) {
        float* cp = static_cast<float*>(p.C) + o;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += bv[e];
        store_f32x8(cp, v, full, p.N - col);
        break;
      }
      // Residual stream: bf16 rows, except the class-token rows (row % tokens
      // == 0), which live in fp32 in ccls when it is given.
      float* cls_row = nullptr;
      if constexpr (E == Epi::BiasResid || E == Epi::Patch) {
        if (p.ccls != nullptr) {
          const int bi = row / p.tokens;
          if (row == bi * p.tokens) cls_row = p.ccls + (int64_t)bi * p.N + col;
        }
      }
      uint16_t* cp = static_cast<uint16_t*>(p.C) + o;
      if constexpr (LN_CONSUMER) {
        // Pre-activation: acc + bias, or with a folded LayerNorm
        // rstd * acc - rstd * mean * colsum + bias.
        if (!CONV && p.ln_in != nullptr) {
          const float2 rs = rowst[pass * SR + rl];
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = fmaf(v[e], rs.x, fmaf(rs.y, cs[e], bv[e]));
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += bv[e];
        }
      }
      if constexpr (E == Epi::BiasGelu) {
        if (p.aux != nullptr)  // keep the pre-activation for the backward
          store_bf16x8(p.aux + (int64_t)row * p.ldaux + col, v, full, p.N - col);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = gelu_poly(v[e]);
      } else if constexpr (E == Epi::GeluBwd) {
        if (full) {
          const u32x4 x = res[it];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] *= gelu_poly_grad(
                __uint_as_float((e & 1) ? (x[e >> 1] & 0xffff0000u) : (x[e >> 1] << 16)));
        } else {
          const uint16_t* ap = p.aux + (int64_t)row * p.ldaux + col;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] = col + e < p.N ? v[e] * gelu_poly_grad(bf16_to_f32(ap[e])) : 0.0f;
        }
      } else if constexpr (E == Epi::BiasResid) {
        if (cls_row != nullptr) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] = col + e < p.N ? cls_row[e] + (v[e] + bv[e]) : 0.0f;
          store_f32x8(cls_row, v, full, p.N - col);
          if (p.ln_out != nullptr) {
            store_bf16x8(cp, v, full, p.N - col);
#pragma unroll
            for (int e = 0; e < 8; ++e) st[e] = v[e];
            st_ok = true;
          }
          break;
        }
        if (full) {
          const u32x4 x = res[it];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] = __uint_as_float((e & 1) ? (x[e >> 1] & 0xffff0000u) : (x[e >> 1] << 16)) +
                   (v[e] + bv[e]);
        } else {
          const uint16_t* rp = p.res != nullptr ? p.res + (int64_t)row * p.ldres + col : cp;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] = col + e < p.N ? bf16_to_f32(rp[e]) + (v[e] + bv[e]) : 0.0f;
        }
      } else if constexpr (E == Epi::Patch) {  // class rows (t == 0) take cls + pos[0], no product
        const int t = row % p.tokens;
        const float* pp = p.pos + (int64_t)t * p.ldpos + col;
        if (full) {
          const f32x4 p0 = *reinterpret_cast<const f32x4*>(pp);
          const f32x4 p1 = *reinterpret_cast<const f32x4*>(pp + 4);
          const float pv[8] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
          if (t == 0) {
            const f32x4 c0 = *reinterpret_cast<const f32x4*>(p.cls + col);
            const f32x4 c1 = *reinterpret_cast<const f32x4*>(p.cls + col + 4);
            const float cv[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = cv[e] + pv[e];
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = (v[e] + bv[e]) + pv[e];
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (col + e < p.N) v[e] = (t == 0 ? p.cls[col + e] : v[e] + bv[e]) + pp[e];
        }
        if (cls_row != nullptr) {
          store_f32x8(cls_row, v, full, p.N - col);
          if (p.ln_out != nullptr) {
            store_bf16x8(cp, v, full, p.N - col);
#pragma unroll
            for (int e = 0; e < 8; ++e) st[e] = v[e];
            st_ok = true;
          }
          break;
        }
      }
      if constexpr (E == Epi::Bias || E == Epi::BiasResid) {
        if (p.relu) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = fmaxf(v[e], 0.0f);
        }
      }
      store_bf16x8(cp, v, full, p.N - col);
      if constexpr (LN_PRODUCER) {  // statistics of the values (before rounding)
#pragma unroll
        for (int e = 0; e < 8; ++e) st[e] = v[e];
        st_ok = true;
      }
      } while (0);
      if constexpr (LN_PRODUCER) {
        if (p.ln_out != nullptr) {
          // Statistics of each 64-column segment: the 8 lanes of an aligned
          // group hold its 8 chunks (N % 8 == 0, so a chunk is whole or
          // absent); three DPP merges give every lane the group's total.
          const LnStat ls = ln_of_group8(st, st_ok, (p.N & 63) == 0);
          const int seg = (n0 >> 6) + (cc >> 3);
          if ((cc & 7) == 0 && 64 * seg < p.N)
            p.ln_out[(int64_t)row * p.ln_ld + seg] = make_float2(ls.n * ls.mean, ls.m2);
        }
      }
    }
    if (pass + 1 < BM / SR) {
      wait_lds();  // staged rows read by every wave before the next pass overwrites them
      __builtin_amdgcn_s_barrier();
    }
  }
}


// Persistent variant for the Bias, BiasGelu and BiasResid epilogues (the
// q/k/v, fc1, projection and fc2 GEMMs of the forward): one 512-thread
// workgroup per CU walks 256x256 tiles v = blockIdx.x + gridDim.x * j (same
// XCD-aware order as above).  Its epilogue is wave-local: each wave converts
// its 128x64 block to bf16 in registers, transposes it through a private
// 32x32 LDS slot (the residual epilogue: 32x16 fp32 values, before the
// residual add and the one rounding) and writes 16-byte row chunks with
// buffer stores.  The epilogue's column vectors come through a second
// per-wave LDS block, loaded at the tile's last K step.  Every wave
// issues exactly 16 stores per tile (rows past M / chunks past N get an offset
// past the buffer's end and are dropped), after the first K step of the next
// tile has been put in flight; the next tile's first wait then leaves those 16
// stores outstanding, so they drain under its main loop instead of stalling
// the CU.  Operands are swapped in the MFMA (D = W A^T) so that a lane holds 4
// consecutive output columns; accumulators live in AGPRs.
// Requirements (checked by the launcher, persistent_ok): a bias, ReLU only on
// the Bias (no folded LayerNorm) and BiasResid epilogues, K % 64 == 0 or (the
// residual epilogue) row strides that cover a ragged last step, N % 8 == 0,
// ldc % 8 == 0 (and ldres % 8 == 0), no aux output, no split K, and with
// class-token rows at least 128 tokens.
constexpr int kPersSlotStride = 72;     // bytes per row of a wave's 32x32 bf16 slot
constexpr int kPersSlotStrideF32 = 80;  // bytes per row of a wave's 32x16 fp32 slot
constexpr int kTilePers = 256;       // rows per persistent tile
// Residual epilogue: 32-row blocks of the residual requested at a tile's last
// K step (1 or 2; the others one block ahead of their use, in a ring of two).
constexpr int kResPre = 1;
// Residual blocks held in registers by the epilogue (a ring): kResRing - 1
// blocks of loads stay in flight ahead of the block being processed.
constexpr int kResRing = 3;

template <Epi E, bool LNF>
__global__ __launch_bounds__(512) void gemm_bf16_persistent(Params p) {
  static_assert(E == Epi::Bias || E == Epi::BiasGelu || E == Epi::BiasResid, "persistent epilogues");
  static_assert(!(LNF && E == Epi::BiasResid), "LayerNorm consumers are Bias / BiasGelu");
  asm volatile("" ::: "a0");  // let the accumulators take AGPRs
  constexpr int BM = 256, BN = 256, WN = 4, NW = 8, WTM = 128, WTN = 64, TM = 4, TN = 2;
  constexpr int STAGE = (BM + BN) * kRowBytes;
  // Epilogue slot per wave: 32 rows x 32 bf16 columns, or (residual epilogue,
  // fp32 staging) 32 rows x 16 fp32 columns.
  constexpr int ES = E == Epi::BiasResid ? kPersSlotStrideF32 : kPersSlotStride, SLOT = 32 * ES;
  constexpr int ROWST = LNF ? 2 * BM * 8 : 0;  // LayerNorm factors of two tiles' rows
  // Per wave 1 KB for the epilogue's column vectors of its 64 columns: the
  // bias, and the folded-LayerNorm column sums or (residual epilogue) the
  // fp32 residual of the class-token row among its 128 rows (below).
  constexpr int AUX = NW * 1024;
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE + NW * SLOT + ROWST + AUX];
  auto bar = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int tiles_m = (p.M + BM - 1) / BM, total = tiles_m * p.tiles_n;
  const int q = total >> 3, r8 = total & 7;
  auto tile_of = [&](int v, int& m0, int& n0) {
    const int xcd = v & 7, idx = v >> 3;
    const int logical = (xcd < r8) ? xcd * (q + 1) + idx : r8 * (q + 1) + (xcd - r8) * q + idx;
    const int gsz = p.group_m * p.tiles_n, group = logical / gsz, in_group = logical - group * gsz;
    const int gm = min(p.group_m, tiles_m - group * p.group_m);
    const int tile_n = in_group / gm, tile_m = group * p.group_m + (in_group - tile_n * gm);
    m0 = tile_m * BM;
    n0 = tile_n * BN;
  };
  // Loads: waves 0-3 bring A rows, waves 4-7 W rows; wave w covers rows
  // (w & 3) * 64 .. +63 of its operand's tile as 8 blocks of 8 rows.  Block i
  // lands at LDS block w * 8 + i (the A tile, then the W tile).  Rows past
  // the end re-read the last row (their results are never stored).
  const int prow = lane >> 3, pcx = (lane & 7) ^ prow;
  const bool loads_a = wave < 4;
  const uint16_t* lsrc = loads_a ? p.A : p.W;
  const int lld = (int)(loads_a ? p.lda : p.ldw);
  const int llim = (loads_a ? p.M : p.N) - 1;
  const int loff = (wave & 3) * 64;
  // K steps; a ragged last step (kpart = K % 64 columns; residual epilogue
  // only) is loaded whole (the operands' row strides reach past it) and its
  // fragments are masked.
  const int nk = (p.K + kBK - 1) / kBK, kpart = p.K % kBK;
  auto load1 = [&](int stage, int r0, int kt, int i, int xl, int pr) {
    const int rb = min(r0 + loff + 8 * i, llim);
    const int rl = min(r0 + loff + 8 * i + pr, llim) - rb;
    const uint32_t off = (uint32_t)(rl * lld + ((xl ^ i) << 3)) * 2u;
    const char* g = reinterpret_cast<const char*>(lsrc + (int64_t)rb * lld + kt * kBK);
    __builtin_amdgcn_global_load_lds((global_void*)(g + off),
                                     (lds_void*)(smem + stage * STAGE + (wave * 8 + i) * 1024), 16,
                                     0, 0);
  };
  const int lr = lane & 31, lg = lane >> 5;
  // LDS byte offset of fragment (quarter kk, block i) in a stage: base ^ (kk << 5).
  int abase[TM], bbase[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = wm * WTM + i * 32 + lr;
    abase[i] = r * kRowBytes + ((lg ^ swz(r)) << 4);
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int r = wn * WTN + j * 32 + lr;
    bbase[j] = BM * kRowBytes + r * kRowBytes + ((lg ^ swz(r)) << 4);
  }
  char* const slot = smem + 2 * STAGE + wave * SLOT;
  float2* const rowst = reinterpret_cast<float2*>(smem + 2 * STAGE + NW * SLOT);
  char* const aux = smem + 2 * STAGE + NW * SLOT + ROWST + wave * 1024;
  // Residual epilogue: lane l holds row rloc = l/2 of each 32-row block of the
  // wave, columns 8 (l%2) .. +7 of each 16-column pass.
  const int rloc = lane >> 1, cloc = (lane & 1) * 8;
  int par = 0;  // half of rowst this tile uses
  int v = blockIdx.x;
  if (v >= total) return;
  int m0, n0;
  tile_of(v, m0, n0);
#pragma unroll
  for (int i = 0; i < 8; ++i) load1(0, loads_a ? m0 : n0, 0, i, pcx, prow);
  int buf = 0;
  bool stores_out = false;
  while (true) {
    const int vn = v + gridDim.x;
    const bool has_next = vn < total;
    int m1 = m0, n1 = n0;
    if (has_next) tile_of(vn, m1, n1);
    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
    // Residual epilogue: the bf16 residual chunks of two 32-row blocks (a
    // ring: block i in slot i % 2), the wave's class-token row (row - wrow0)
    // and its image.
    u32x4 rz[kResRing][TN][2];
    int cls_rel = -1, cls_b = 0;
    // Residual block i of this lane (rows of the wave as one buffer range:
    // rows past M read as zeros and are never stored).
    auto load_res = [&](int i, u32x4 (&dst)[TN][2]) {
      const uint16_t* rsrc = p.res != nullptr ? p.res : static_cast<const uint16_t*>(p.C);
      const int rld = (int)(p.res != nullptr ? p.ldres : p.ldc);
      const int wr0 = __builtin_amdgcn_readfirstlane(m0 + wm * WTM);
      const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(rsrc) + (int64_t)wr0 * rld, (short)0,
          __builtin_amdgcn_readfirstlane(max(0, min(WTM, p.M - wr0)) * rld * 2), kRsrcWord3);
      const int cb = min(n0 + wn * WTN + cloc, p.N - 8);
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int c = min(cb + j * 32 + h * 16, p.N - 8);
          dst[j][h] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(rr, ((rloc + i * 32) * rld + c) * 2, 0, 0));
        }
    };
    // Residual epilogue: the wave's class-token row, and the request of the
    // epilogue's operands at the tile's last K step (below).
    if constexpr (E == Epi::BiasResid) {
      const int wrow0 = m0 + wm * WTM;
      if (p.ccls != nullptr) {
        const int bi = (wrow0 + p.tokens - 1) / p.tokens, rc = bi * p.tokens;
        if (rc < wrow0 + WTM && rc < p.M) {
          cls_rel = rc - wrow0;
          cls_b = bi;
        }
      }
    }
    // The epilogue's operands, requested at the tile's last K step (ahead of
    // that step's tile loads): residual epilogue, the first residual blocks
    // (registers); every epilogue, by one direct load into this wave's LDS
    // block, the bias of its 64 columns (lanes 0-15, bytes 0-255) and the
    // folded-LayerNorm column sums or the class-token row's fp32 residual
    // (lanes 16-31, bytes 256-511; lanes 32-63 repeat lanes 0-31).
    auto epi_request = [&]() {
      if constexpr (E == Epi::BiasResid) {
#pragma unroll
        for (int i = 0; i < kResPre; ++i) load_res(i, rz[i % kResRing]);
      }
      const int l = lane & 31, c = min(n0 + wn * WTN + 4 * (l & 15), p.N - 4);
      const float* src = p.bias + c;
      if (l >= 16) {
        if constexpr (E == Epi::BiasResid) {
          if (cls_rel >= 0) src = p.ccls + (int64_t)cls_b * p.N + c;
        } else if constexpr (LNF) {
          src = p.ln_colsum + c;
        }
      }
      __builtin_amdgcn_global_load_lds((global_void*)src, (lds_void*)aux, 16, 0, 0);
    };
    {
      // Fragments of two K quarters in flight: a quarter's MFMAs run while the
      // LDS reads of the next quarter are issued between them, so a wave never
      // waits on reads issued just before.  A step's last quarter is
      // multiplied after the next step's barrier (the stage it came from may
      // be overwritten only after that barrier, and its fragments are already
      // in registers), behind that step's first reads.  Every step issues its
      // eight tile loads (the last step of the last tile re-reads its own first
      // step into the idle stage), so each quarter is one straight-line block.
      bf16x8 fa[2][TM], fb[2][TN];
      // Ragged last step: zero both operands' elements at k >= K (this lane's
      // fragments of quarter kk hold k = 16 kk + 8 lg .. +7 of the step), so
      // that whatever lies past K in the rows never enters a product.
      auto mask_tail = [&](bf16x8* fa_, bf16x8* fb_, int kk) {
        const int k0 = 16 * kk + 8 * lg;
        u32x4 m;
  #pragma unroll
        for (int d = 0; d < 4; ++d)
          m[d] = (k0 + 2 * d < kpart ? 0x0000ffffu : 0u) | (k0 + 2 * d + 1 < kpart ? 0xffff0000u : 0u);
  #pragma unroll
        for (int i = 0; i < TM; ++i) fa_[i] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, fa_[i]) & m);
  #pragma unroll
        for (int j = 0; j < TN; ++j) fb_[j] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, fb_[j]) & m);
      };
  #define ELASTO_PERS_STEP(FIRST)                                                              \
      {                                                                                        \
        if ((FIRST) && stores_out) wait_vm_lds<16>();                                          \
        else wait_vm_lds<0>();                                                                 \
        __builtin_amdgcn_s_barrier();                                                          \
        __builtin_amdgcn_sched_barrier(0);                                                     \
        LnStat lst{0.0f, 0.0f, 0.0f};                                                          \
        if (LNF && (FIRST))                                                                    \
          ln_sums(p.ln_in + (int64_t)min(m0 + (tid >> 1), p.M - 1) * p.ln_ld, p.K, tid & 1, 2, \
                  lst);                                                                        \
        const bool more = kt + 1 < nk;                                                         \
        if (!more) epi_request();                                                              \
        const int nr0 = more ? (loads_a ? m0 : n0) : (loads_a ? m1 : n1), nkt = more ? kt + 1 : 0; \
        const int so = buf * STAGE;                                                            \
        int xl = pcx, pr = prow, ab[TM], bb[TN];                                               \
        _Pragma("unroll") for (int i = 0; i < TM; ++i) ab[i] = abase[i];                       \
        _Pragma("unroll") for (int j = 0; j < TN; ++j) bb[j] = bbase[j];                       \
        asm volatile("" : "+v"(xl), "+v"(pr));                                                 \
        _Pragma("unroll") for (int i = 0; i < TM; ++i) asm volatile("" : "+v"(ab[i]));         \
        _Pragma("unroll") for (int j = 0; j < TN; ++j) asm volatile("" : "+v"(bb[j]));         \
        _Pragma("unroll") for (int kk = 0; kk < kBK / 16; ++kk) {                              \
          const int rs = kk & 1, ms = rs ^ 1, kx = kk << 5;                                    \
          _Pragma("unroll") for (int i = 0; i < TM; ++i)                                       \
            fa[rs][i] = *reinterpret_cast<const bf16x8*>(smem + ((ab[i] + so) ^ kx));          \
          _Pragma("unroll") for (int j = 0; j < TN; ++j)                                       \
            fb[rs][j] = *reinterpret_cast<const bf16x8*>(smem + ((bb[j] + so) ^ kx));          \
          if (E == Epi::BiasResid && kpart != 0 && !more) mask_tail(fa[rs], fb[rs], kk);       \
          if (kk < 3) {                                                                        \
            _Pragma("unroll") for (int t = (8 * kk + 2) / 3; t < (8 * (kk + 1) + 2) / 3; ++t)  \
              load1(buf ^ 1, nr0, nkt, t, xl, pr);                                             \
          }                                                                                    \
          if (!((FIRST) && kk == 0)) {                                                         \
            _Pragma("unroll") for (int i = 0; i < TM; ++i)                                     \
            _Pragma("unroll") for (int j = 0; j < TN; ++j)                                     \
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[ms][j], fa[ms][i],        \
                                                                  acc[i][j], 0, 0, 0);         \
            _Pragma("unroll") for (int t = 0; t < 6; ++t) {                                    \
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                               \
              __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);                               \
            }                                                                                  \
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);                                 \
          }                                                                                    \
          __builtin_amdgcn_sched_barrier(0);                                                   \
        }                                                                                      \
        if (LNF && (FIRST)) {                                                                  \
          ln_merge_dpp<kDppXor1>(lst);                                                         \
          if ((tid & 1) == 0) rowst[par * BM + (tid >> 1)] = ln_factors(lst, p.ln_eps);        \
        }                                                                                      \
        buf ^= 1;                                                                              \
      }
      {
        const int kt = 0;
        ELASTO_PERS_STEP(true)
      }
  #pragma clang loop unroll(disable)
      for (int kt = 1; kt < nk; ++kt) ELASTO_PERS_STEP(false)
  #undef ELASTO_PERS_STEP
      // The tile's last quarter.
  #pragma unroll
      for (int i = 0; i < TM; ++i)
  #pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[1][j], fa[1][i], acc[i][j], 0, 0, 0);
    }
    if constexpr (LNF) {
      if (nk == 1) {  // no later step barrier in this tile
        wait_lds();
        bar();
      }
    }

    // Epilogue.  acc[i][j][e] is output row m0 + wm*128 + i*32 + lr, column
    // n0 + wn*64 + j*32 + 8*(e/4) + 4*lg + e%4.
    const int rows_valid = min(BM, p.M - m0);
    const int nrec = rows_valid * (int)p.ldc * 2;
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        static_cast<uint16_t*>(p.C) + (int64_t)m0 * p.ldc, (short)0, nrec, kRsrcWord3);
    // The column vectors in the wave's LDS block hold columns
    // n0 + wn*64 + 4q .. +3 at 16q, clamped into [0, N) (the columns past N
    // are computed from re-read rows and never stored).
    if constexpr (E == Epi::BiasResid) {
      // C = residual + acc + bias: fp32 staging of acc + bias, 16 columns per
      // pass (i, j, h); lane l then holds row r = l/2 of the 32-row block,
      // columns 8 (l%2) .. +7 of the pass.  The residual comes from res (or C
      // in place), except on the class-token rows (row % tokens == 0) when
      // ccls is given: there it is the fp32 ccls row, which takes the fp32
      // result (and C its bf16 rounding when the LayerNorm statistics are
      // produced).  Everything the epilogue reads was requested at the last
      // K step: wait for it (the next tile's first-step loads, issued after
      // it, may stay in flight).
      wait_vm_lds<8>();
      asm volatile("" ::: "memory");
      const int row_l0 = m0 + wm * WTM + rloc;  // this lane's row in block i: row_l0 + 32 i
      const int cls_i = (cls_rel >= 0 && (cls_rel & 31) == rloc) ? cls_rel >> 5 : -1;
      const int seg = (n0 + wn * WTN) >> 6;  // this wave's 64 columns: one statistics segment
      const int wo = lr * ES + lg * 16, ro = rloc * ES + (lane & 1) * 32;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        // Keep kResRing - 1 blocks ahead in flight (slot of block i - 1 is free).
        if (i == 0) {
#pragma unroll
          for (int b = kResPre; b < kResRing - 1 && b < TM; ++b) load_res(b, rz[b % kResRing]);
        }
        if (i + kResRing - 1 >= kResPre && i + kResRing - 1 < TM)
          load_res(i + kResRing - 1, rz[(i + kResRing - 1) % kResRing]);
        const int row = row_l0 + i * 32;
        const bool row_ok = row < p.M, cls = i == cls_i;
        // Statistics of the lane's four chunks of the segment: pairwise
        // merges of equal sizes when N is a multiple of 64 (every chunk of a
        // segment inside [0, N) whole), else one at a time.
        static_assert(TN == 2, "segment = two 32-column blocks");
        const bool whole = (p.N & 63) == 0;
        LnStat ls{0.0f, 0.0f, 0.0f}, lj{0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int gg = 0; gg < 2; ++gg) {
              const int g = 2 * h + gg;
              // Bias of columns j*32 + 8g + 4lg .. +3 of the wave's 64.
              const f32x4 bv = *reinterpret_cast<const f32x4*>(aux + (j * 32 + 8 * g + 4 * lg) * 4);
              const f32x4 w = {acc[i][j][4 * g] + bv[0], acc[i][j][4 * g + 1] + bv[1],
                               acc[i][j][4 * g + 2] + bv[2], acc[i][j][4 * g + 3] + bv[3]};
              *reinterpret_cast<f32x4*>(slot + wo + gg * 32) = w;
            }
            wait_lds();
            const f32x4 s0 = *reinterpret_cast<const f32x4*>(slot + ro);
            const f32x4 s1 = *reinterpret_cast<const f32x4*>(slot + ro + 16);
            const int col = n0 + wn * WTN + j * 32 + h * 16 + cloc;
            const bool ok = row_ok && col + 8 <= p.N;
            float v[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
            if (cls) {
              const char* cr = aux + 256 + (j * 32 + h * 16 + cloc) * 4;
              const f32x4 c0 = *reinterpret_cast<const f32x4*>(cr);
              const f32x4 c1 = *reinterpret_cast<const f32x4*>(cr + 16);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                v[e] += c0[e];
                v[4 + e] += c1[e];
              }
              if (ok) {
                float* cp = p.ccls + (int64_t)cls_b * p.N + col;
                *reinterpret_cast<f32x4*>(cp) = f32x4{v[0], v[1], v[2], v[3]};
                *reinterpret_cast<f32x4*>(cp + 4) = f32x4{v[4], v[5], v[6], v[7]};
              }
            } else {
              const u32x4 x = rz[i % kResRing][j][h];
#pragma unroll
              for (int e = 0; e < 8; ++e)
                v[e] += __uint_as_float((e & 1) ? (x[e >> 1] & 0xffff0000u) : (x[e >> 1] << 16));
              if (p.relu) {
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = fmaxf(v[e], 0.0f);
              }
            }
            u32x4 w;
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2)
              w[q2] = pack_bf16x2(v[2 * q2], v[2 * q2 + 1]);
            const bool st = ok && (!cls || p.ln_out != nullptr);
            __builtin_amdgcn_raw_buffer_store_b128(
                w, rc, st ? ((row - m0) * (int)p.ldc + col) * 2 : nrec, 0, 0);
            const LnStat l8 = ln_of8(v, ok);
            if (whole) {
              if (h == 0) {
                lj = l8;
              } else {
                ln_merge_equal(lj, l8.mean, l8.m2);
                if (j == 0)
                  ls = lj;
                else
                  ln_merge_equal(ls, lj.mean, lj.m2);
              }
            } else {
              ln_merge(ls, l8.n, l8.mean, l8.m2);
            }
            wait_lds();  // the slot is rewritten by the next pass
          }
        if (p.ln_out != nullptr) {  // this row's 64-column segment: lanes l and l ^ 1
          if (whole)
            ln_merge_dpp_equal<kDppXor1>(ls);
          else
            ln_merge_dpp<kDppXor1>(ls);
          if ((lane & 1) == 0 && row_ok && 64 * seg < p.N)
            p.ln_out[(int64_t)row * p.ln_ld + seg] = make_float2(ls.n * ls.mean, ls.m2);
        }
      }
    } else {
      // Folded LayerNorm: (rstd, -rstd * mean) of this lane's 4 rows.
      float2 rs[TM];
      if constexpr (LNF) {
  #pragma unroll
        for (int i = 0; i < TM; ++i) rs[i] = rowst[par * BM + wm * WTM + i * 32 + lr];
      }
      const int lane_st = ((wm * WTM + (lane >> 2)) * (int)p.ldc + n0 + wn * WTN + (lane & 3) * 8) * 2;
      const int wofs = lr * ES + lg * 8, rofs = (lane >> 2) * ES + (lane & 3) * 16;
      // The column vectors were requested at the last K step (the next tile's
      // first-step loads, issued after them, may stay in flight).
      wait_vm_lds<8>();
      asm volatile("" ::: "memory");
      // Row blocks outermost: the two 64-byte halves of a wave's 128-byte row
      // segment are stored one pass apart.
  #pragma unroll
      for (int i = 0; i < TM; ++i) {
  #pragma unroll
        for (int j = 0; j < TN; ++j) {
        int lst = lane_st, wo = wofs, ro = rofs;
        asm volatile("" : "+v"(lst), "+v"(wo), "+v"(ro));
  #pragma unroll
          for (int g = 0; g < 4; ++g) {
            // Bias (and column sums) of columns j*32 + 8g + 4lg .. +3 of the wave's 64.
            const int vo = (j * 32 + 8 * g + 4 * lg) * 4;
            const f32x4 bv = *reinterpret_cast<const f32x4*>(aux + vo);
            f32x4 cs;
            if constexpr (LNF) cs = *reinterpret_cast<const f32x4*>(aux + 256 + vo);
            float t[4];
  #pragma unroll
            for (int e = 0; e < 4; ++e) {
              if constexpr (LNF)
                t[e] = fmaf(acc[i][j][4 * g + e], rs[i].x, fmaf(rs[i].y, cs[e], bv[e]));
              else
                t[e] = acc[i][j][4 * g + e] + bv[e];
              if constexpr (E == Epi::BiasGelu) t[e] = gelu_poly(t[e]);
              if constexpr (E == Epi::Bias && !LNF) {
                if (p.relu) t[e] = fmaxf(t[e], 0.0f);
              }
            }
            u32x2 w;
            w[0] = pack_bf16x2(t[0], t[1]);
            w[1] = pack_bf16x2(t[2], t[3]);
            *reinterpret_cast<u32x2*>(slot + wo + g * 16) = w;
          }
          wait_lds();
  #pragma unroll
          for (int h = 0; h < 2; ++h) {
            const u32x2 lo = *reinterpret_cast<const u32x2*>(slot + ro + h * 16 * ES);
            const u32x2 hi = *reinterpret_cast<const u32x2*>(slot + ro + h * 16 * ES + 8);
            const int rl = wm * WTM + i * 32 + h * 16 + (lane >> 2);
            const int col = n0 + wn * WTN + j * 32 + (lane & 3) * 8;
            const bool ok = rl < rows_valid && col + 8 <= p.N;
            const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
            __builtin_amdgcn_raw_buffer_store_b128(
                w, rc, ok ? lst + (i * 32 + h * 16) * (int)p.ldc * 2 + j * 64 : nrec, 0, 0);
          }
          wait_lds();  // the slot is rewritten by the next block
        }
      }
    }
    if (!has_next) break;
    v = vn;
    m0 = m1;
    n0 = n1;
    stores_out = true;
    par ^= 1;
  }
  // The last step issued loads into the idle stage: let them land before the
  // wave ends.
  wait_vm_lds<0>();
}

// Split-K epilogue.  A GEMM whose tiles would occupy few of the CUs (small M:
// batch-1 and batch-8 forwards) runs as ksplit K-chunks of the BiasF32 kernel
// writing fp32 partial products, then this kernel sums each output's partials
// in chunk order and applies the epilogue E: the folded-LayerNorm consumer
// (Bias, BiasGelu) or the residual add with the LayerNorm-statistics producer
// (BiasResid), with the same arithmetic as the tile epilogues.  One thread per
// 8-column chunk of an output row; a row's chunks are padded to a multiple of
// 8 threads, so the 8 lanes of an aligned group hold one 64-column segment.
struct SplitEpi {
  const float* part;   // ksplit slices of [M][ldp] fp32
  int64_t ldp, slice;  // row stride of a slice (a multiple of 8), elements per slice
  int ksplit, M, N, K, cpr;
  void* C;
  int64_t ldc;
  const float* bias;
  const uint16_t* res;  // BiasResid residual (nullptr: C)
  int64_t ldres;
  float* ccls;
  int tokens;
  float2* ln_out;
  const float2* ln_in;
  int64_t ln_ld;
  const float* ln_colsum;
  float ln_eps;
};

template <Epi E>
__global__ __launch_bounds__(64) void splitk_epilogue_kernel(SplitEpi q) {
  static_assert(E == Epi::Bias || E == Epi::BiasGelu || E == Epi::BiasResid, "split-K epilogues");
  const int64_t g = (int64_t)blockIdx.x * 64 + threadIdx.x;
  const int row = (int)(g / q.cpr), cc = (int)(g - (int64_t)row * q.cpr);
  // Folded LayerNorm: the factors of each row the block touches (at most
  // 64 / 8 + 1 rows: cpr >= 8), merged once per row by one lane, not by
  // every thread of the row.
  float2 rs = make_float2(0.0f, 0.0f);
  if constexpr (E == Epi::Bias || E == Epi::BiasGelu) {
    if (q.ln_in != nullptr) {
      __shared__ float2 fac[64 / 8 + 1];
      const int r0 = (int)((int64_t)blockIdx.x * 64 / q.cpr);
      const int r = r0 + (int)threadIdx.x;
      if (threadIdx.x <= 64 / 8 && r < q.M && (int64_t)r * q.cpr < (int64_t)blockIdx.x * 64 + 64) {
        LnStat st{0.0f, 0.0f, 0.0f};
        ln_sums(q.ln_in + (int64_t)r * q.ln_ld, q.K, 0, 1, st);
        fac[threadIdx.x] = ln_factors(st, q.ln_eps);
      }
      __syncthreads();
      if (row < q.M) rs = fac[row - r0];
    }
  }
  if (row >= q.M) return;  // whole 8-lane groups: cpr is a multiple of 8
  const int col = cc * 8;
  const bool col_in = col < q.N, full = col + 8 <= q.N;
  float v[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  if (col_in) {
    const float* pp = q.part + (int64_t)row * q.ldp + col;
    for (int c0 = 0; c0 < q.ksplit; c0 += 8) {
      f32x4 t[8][2];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float* src = pp + (int64_t)min(c0 + u, q.ksplit - 1) * q.slice;
        t[u][0] = *reinterpret_cast<const f32x4*>(src);
        t[u][1] = *reinterpret_cast<const f32x4*>(src + 4);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (c0 + u < q.ksplit) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] += t[u][0][e];
            v[4 + e] += t[u][1][e];
          }
        }
    }
  }
  float bv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bv[e] = col + e < q.N ? q.bias[col + e] : 0.0f;
  uint16_t* cp = static_cast<uint16_t*>(q.C) + (int64_t)row * q.ldc + col;
  if constexpr (E == Epi::Bias || E == Epi::BiasGelu) {
    if (!col_in) return;
    if (q.ln_in != nullptr) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float cs = col + e < q.N ? q.ln_colsum[col + e] : 0.0f;
        v[e] = fmaf(v[e], rs.x, fmaf(rs.y, cs, bv[e]));
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += bv[e];
    }
    if constexpr (E == Epi::BiasGelu) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = gelu_poly(v[e]);
    }
    store_bf16x8(cp, v, full, q.N - col);
  } else {
    float st[8];
    bool st_ok = false;
    if (col_in) {
      float* cls_row = nullptr;
      if (q.ccls != nullptr) {
        const int bi = row / q.tokens;
        if (row == bi * q.tokens) cls_row = q.ccls + (int64_t)bi * q.N + col;
      }
      if (cls_row != nullptr) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = col + e < q.N ? cls_row[e] + (v[e] + bv[e]) : 0.0f;
        store_f32x8(cls_row, v, full, q.N - col);
        if (q.ln_out != nullptr) store_bf16x8(cp, v, full, q.N - col);
      } else {
        const uint16_t* rp = q.res != nullptr ? q.res + (int64_t)row * q.ldres + col : cp;
        if (full) {
          const u32x4 x = *reinterpret_cast<const u32x4*>(rp);
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] = __uint_as_float((e & 1) ? (x[e >> 1] & 0xffff0000u) : (x[e >> 1] << 16)) +
                   (v[e] + bv[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] = col + e < q.N ? bf16_to_f32(rp[e]) + (v[e] + bv[e]) : 0.0f;
        }
        store_bf16x8(cp, v, full, q.N - col);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) st[e] = v[e];
      st_ok = true;
    }
    if (q.ln_out != nullptr) {
      const LnStat ls = ln_of_group8(st, st_ok, (q.N & 63) == 0);
      const int seg = cc >> 3;
      if ((cc & 7) == 0 && 64 * seg < q.N)
        q.ln_out[(int64_t)row * q.ln_ld + seg] = make_float2(ls.n * ls.mean, ls.m2);
    }
  }
}

template <int BM, int BN, int WM, int WN, Epi E, bool CONV, int STAGES = 2>
hipError_t launch_cfg(const Params& p0, int row0, hipStream_t s) {
  Params p = p0;
  p.row0 = row0;
  const int64_t tm = (p.M - row0 + BM - 1) / BM, tn = (p.N + BN - 1) / BN;
  p.tiles_n = (int)tn;
  // Long K: tiles in flight stream whole A panels, so few panels per group
  // keep each panel's N tiles together; short K: a wider group.
  p.group_m = p.K >= 2048 ? 2 : 4;
  const int64_t blocks = tm * tn;
  if (blocks <= 0) return hipSuccess;
  const bool ln_consumer = (E == Epi::Bias || E == Epi::BiasGelu) && !CONV && p.ln_in != nullptr;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, E, CONV, STAGES>),
                     dim3((unsigned)blocks, (unsigned)(p.ksplit > 1 ? p.ksplit : 1)),
                     dim3(64 * WM * WN), ln_consumer ? BM * 8 : 0, s, p);
  return hipGetLastError();
}

// Compute units of the current device (cached per device).
int device_cus() {
  static int cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

template <Epi E>
bool persistent_ok(const Params& p) {
  if constexpr (E != Epi::Bias && E != Epi::BiasGelu && E != Epi::BiasResid) {
    return false;
  } else {
    if (E == Epi::BiasResid && p.res != nullptr && p.ldres % 8 != 0) return false;
    // A wave's 128 rows may hold one class-token row (its fp32 residual is
    // staged in the wave's LDS block).
    if (E == Epi::BiasResid && p.ccls != nullptr && p.tokens < 128) return false;
    // K: whole 64-column steps, or (residual GEMMs: fc2 of narrow modes) a
    // ragged last step that the operands' row strides cover (it is loaded
    // whole and masked in registers).
    const int64_t kpad = (p.K + kBK - 1) / kBK * kBK;
    const bool k_ok = p.K % kBK == 0 || (E == Epi::BiasResid && p.lda >= kpad && p.ldw >= kpad);
    // ReLU (convolution blocks): on the Bias and BiasResid epilogues, not on
    // a folded-LayerNorm consumer.
    const bool relu_ok = !p.relu || (E != Epi::BiasGelu && p.ln_in == nullptr);
    return p.bias != nullptr && relu_ok && p.aux == nullptr && p.ksplit <= 1 && p.K >= 1 && k_ok &&
           p.N % 8 == 0 &&
           p.ldc % 8 == 0 && (int64_t)kTilePers * p.ldc * 2 < ((int64_t)1 << 31);
  }
}

// Whether the planner (plan 0) takes the persistent kernel for a whole
// launch: for the residual GEMMs only with short K (the projection), where
// the epilogue is a large share of a tile; a split plan's head and the forced
// plan 6 run it wherever persistent_ok holds.
template <Epi E>
bool persistent_default(const Params& p) {
  return persistent_ok<E>(p) && (E != Epi::BiasResid || p.K <= 1024);
}

// Rows [0, rows) of the 256x256 tiling with the persistent kernel.
template <Epi E>
hipError_t launch_persistent(const Params& p0, int rows, hipStream_t s) {
  if constexpr (E != Epi::Bias && E != Epi::BiasGelu && E != Epi::BiasResid) {
    return hipErrorInvalidValue;
  } else {
    Params p = p0;
    p.M = rows;
    p.row0 = 0;
    p.tiles_n = (p.N + 255) / 256;
    // Row panels per group of the tile order: measured best at 8 for outputs of
    // at most 9 tiles across (q/k/v), 4 for wider ones (fc1); the residual
    // GEMMs keep the non-persistent kernel's choice.
    if (E == Epi::BiasResid)
      p.group_m = p.K >= 2048 ? 2 : 4;
    else
      p.group_m = p.tiles_n <= 9 ? 8 : 4;
    const int64_t tiles = (int64_t)((rows + 255) / 256) * p.tiles_n;
    if (tiles <= 0) return hipSuccess;
    const int grid = (int)std::min<int64_t>(tiles, device_cus());
    if constexpr (E == Epi::BiasResid) {
      hipLaunchKernelGGL((gemm_bf16_persistent<E, false>), dim3(grid), dim3(512), 0, s, p);
    } else {
      if (p.ln_in != nullptr)
        hipLaunchKernelGGL((gemm_bf16_persistent<E, true>), dim3(grid), dim3(512), 0, s, p);
      else
        hipLaunchKernelGGL((gemm_bf16_persistent<E, false>), dim3(grid), dim3(512), 0, s, p);
    }
    return hipGetLastError();
  }
}

// One launch of the tile plan p.plan (see kTilePlans).
template <Epi E, bool CONV>
hipError_t launch_forced(const Params& p, hipStream_t s) {
  switch (p.plan) {
    case 1: return launch_cfg<256, 256, 2, 4, E, CONV>(p, 0, s);
    case 2: return launch_cfg<256, 128, 2, 2, E, CONV>(p, 0, s);
    case 3: return launch_cfg<128, 128, 2, 2, E, CONV>(p, 0, s);
    case 4: return launch_cfg<256, 64, 4, 1, E, CONV>(p, 0, s);
    case 5:
      if constexpr (!CONV && (E == Epi::Bias || E == Epi::BiasGelu || E == Epi::BiasResid)) {
        if (p.K % kBK == 0 && p.K / kBK >= 4) return launch_cfg<128, 128, 2, 2, E, CONV, 4>(p, 0, s);
      }
      return hipErrorNotSupported;
    case 6:
      if constexpr (!CONV) {
        if (persistent_ok<E>(p)) return launch_persistent<E>(p, p.M, s);
      }
      return hipErrorNotSupported;
    default:
      // Split-K plans (7 and up) apply to small-M bf16 GEMMs only
      // (launch_gemm_bf16 takes them before this point).
      return p.plan < kTilePlans ? hipErrorNotSupported : hipErrorInvalidValue;
  }
}

template <Epi E, bool CONV = false>
hipError_t launch_epi(const Params& p, hipStream_t s) {
  if (p.plan != 0) return launch_forced<E, CONV>(p, s);
  // Pick the launch plan that keeps the chip busiest.  Estimated time is the
  // number of rounds of concurrent workgroups (one per CU) times the relative
  // cost of one tile.  Besides single launches of one tile shape there is a
  // split plan against wave quantisation: the whole rounds of 256x256 tiles
  // first, then the remaining row panels as 128x256 or 128x128 tiles
  // (whichever takes fewer tile-weighted rounds) in a second launch.
  constexpr int kCUs = 256;
  constexpr double kRel128x256 = 0.6, kRel128x128 = 0.36;
  auto rounds = [](int64_t tiles) { return (double)((tiles + kCUs - 1) / kCUs); };
  struct Cfg { int bm, bn; double rel; };
  // 256x64 (four waves stacked along M) only for outputs at most 64 wide,
  // where wider tiles would leave half their columns idle.
  const Cfg cfgs[4] = {{256, 256, 1.0}, {256, 128, 0.62}, {128, 128, 0.36}, {256, 64, 0.3}};
  const int ncfg = p.N <= 64 ? 4 : 3;
  int best = 0;
  double best_t = 1e300;
  for (int i = 0; i < ncfg; ++i) {
    const int64_t tiles = ((p.M + cfgs[i].bm - 1) / cfgs[i].bm) * ((p.N + cfgs[i].bn - 1) / cfgs[i].bn);
    const double t = rounds(tiles) * cfgs[i].rel;
    if (t < best_t - 1e-9) { best_t = t; best = i; }
  }
  const int64_t tn = (p.N + 255) / 256, total = tn * ((p.M + 255) / 256);
  const int64_t head_rows = (total / kCUs) * kCUs / tn * 256;  // rows in whole rounds
  if (head_rows > 0 && head_rows < p.M) {
    const int64_t tail_panels = (p.M - head_rows + 127) / 128;
    const double t_wide = kRel128x256 * rounds(tail_panels * tn);
    const double t_sq = kRel128x128 * rounds(tail_panels * ((p.N + 127) / 128));
    const double t = rounds(head_rows / 256 * tn) + std::min(t_wide, t_sq);
    if (t < best_t - 0.1) {
      Params head = p;
      head.M = (int)head_rows;
      // (the head's tiles are whole rounds: persistent at any K)
      hipError_t e = (!CONV && persistent_ok<E>(p))
                         ? launch_persistent<E>(p, (int)head_rows, s)
                         : launch_cfg<256, 256, 2, 4, E, CONV>(head, 0, s);
      if (e != hipSuccess) return e;
      if (t_sq < t_wide - 1e-9) {
        // One round or less of square tiles: the K chains are the critical path.
        if constexpr (!CONV && (E == Epi::Bias || E == Epi::BiasGelu || E == Epi::BiasResid)) {
          if (tail_panels * ((p.N + 127) / 128) < kCUs && p.K % kBK == 0 && p.K / kBK >= 4)
            return launch_cfg<128, 128, 2, 2, E, CONV, 4>(p, (int)head_rows, s);
        }
        return launch_cfg<128, 128, 2, 2, E, CONV>(p, (int)head_rows, s);
      }
      return launch_cfg<128, 256, 2, 4, E, CONV>(p, (int)head_rows, s);
    }
  }
  switch (best) {
    case 0:
      if (!CONV && persistent_default<E>(p)) return launch_persistent<E>(p, p.M, s);
      return launch_cfg<256, 256, 2, 4, E, CONV>(p, 0, s);
    case 1: return launch_cfg<256, 128, 2, 2, E, CONV>(p, 0, s);
    case 2:
      // Less than a round of tiles: each workgroup's K chain is the critical
      // path, so keep three steps of loads in flight.
      if constexpr (!CONV && (E == Epi::Bias || E == Epi::BiasGelu || E == Epi::BiasResid)) {
        const int64_t tiles = ((p.M + 127) / 128) * ((p.N + 127) / 128);
        if (tiles < kCUs && p.K % kBK == 0 && p.K / kBK >= 4)
          return launch_cfg<128, 128, 2, 2, E, CONV, 4>(p, 0, s);
      }
      return launch_cfg<128, 128, 2, 2, E, CONV>(p, 0, s);
    default: return launch_cfg<256, 64, 4, 1, E, CONV>(p, 0, s);
  }
}

// Split-K plan for launches whose 128x128 tiles would fill under half the
// CUs: the K loop is then the critical path of every workgroup (about one
// memory latency per K step).  Cutting it into chunks costs a second launch
// and the fp32 partials' round trip, so the plan takes the chunk count with
// the smallest estimated time, in microseconds, measured on MI355X at batch 1
// and 8 of ViT-B/16:
//   one launch:  3 + 1.1 nk,
//   c chunks:   11 + 1.1 ceil(nk / c) + c M N 8 bytes / 3.5 TB/s,
// with at least two K steps a chunk and at most one workgroup per CU.
// Returns the chunk count (1: no split) and the chunk length.
int split_plan(const Params& p, int64_t ws_bytes, int* kchunk) {
  constexpr int kCUs = 256;
  const int64_t tiles = (int64_t)((p.M + 127) / 128) * ((p.N + 127) / 128);
  const int nk = (p.K + kBK - 1) / kBK;
  if (tiles * 2 > kCUs || nk < 4) return 1;
  const int64_t ldp = (p.N + 7) / 8 * 8;
  const int most = (int)std::min<int64_t>(kCUs / tiles, nk / 2);
  double best_t = 3.0 + 1.1 * nk - 1.0;  // a split must win by a microsecond
  int best = 1;
  for (int c = 2; c <= most; ++c) {
    if ((int64_t)c * p.M * ldp * 4 > ws_bytes) break;
    const int steps = (nk + c - 1) / c;
    const double t = 11.0 + 1.1 * steps + (double)c * p.M * ldp * 8.0 / 3.5e6;
    if (t < best_t) { best_t = t; best = c; }
  }
  if (best < 2) return 1;
  const int steps = (nk + best - 1) / best;
  *kchunk = steps * kBK;
  return (nk + steps - 1) / steps;
}

// A forced split into about `chunks` K-chunks (split plans): only where the
// planner could split (the 128x128 tiles fill under half the CUs), with at
// least two chunks and the partials within the workspace.  Returns the chunk
// count (1: not applicable) and the chunk length.
int forced_split(const Params& p, int64_t ws_bytes, int chunks, int* kchunk) {
  constexpr int kCUs = 256;
  const int64_t tiles = (int64_t)((p.M + 127) / 128) * ((p.N + 127) / 128);
  const int nk = (p.K + kBK - 1) / kBK;
  if (tiles * 2 > kCUs || chunks < 2 || nk < 2) return 1;
  const int steps = (nk + chunks - 1) / chunks;
  const int c = (nk + steps - 1) / steps;
  const int64_t ldp = (p.N + 7) / 8 * 8;
  if (c < 2 || (int64_t)c * p.M * ldp * 4 > ws_bytes) return 1;
  *kchunk = steps * kBK;
  return c;
}

template <Epi E>
hipError_t launch_split(const Params& p, float* ws, int ksplit, int kchunk, hipStream_t s) {
  Params pp = p;
  const int64_t ldp = (p.N + 7) / 8 * 8;
  pp.C = ws;
  pp.ldc = ldp;
  pp.bias = nullptr;
  pp.ccls = nullptr;
  pp.res = nullptr;
  pp.aux = nullptr;
  pp.ln_out = nullptr;
  pp.ln_in = nullptr;
  pp.relu = 0;
  pp.ksplit = ksplit;
  pp.kchunk = kchunk;
  pp.c_split = (int64_t)p.M * ldp;
  hipError_t e = (p.K % kBK == 0 && kchunk / kBK >= 4)
                     ? launch_cfg<128, 128, 2, 2, Epi::BiasF32, false, 4>(pp, 0, s)
                     : launch_cfg<128, 128, 2, 2, Epi::BiasF32, false>(pp, 0, s);
  if (e != hipSuccess) return e;
  SplitEpi q;
  q.part = ws;
  q.ldp = ldp;
  q.slice = pp.c_split;
  q.ksplit = ksplit;
  q.M = p.M;
  q.N = p.N;
  q.K = p.K;
  q.cpr = (int)((p.N + 63) / 64 * 8);
  q.C = p.C;
  q.ldc = p.ldc;
  q.bias = p.bias;
  q.res = p.res;
  q.ldres = p.ldres;
  q.ccls = p.ccls;
  q.tokens = p.tokens;
  q.ln_out = p.ln_out;
  q.ln_in = p.ln_in;
  q.ln_ld = p.ln_ld;
  q.ln_colsum = p.ln_colsum;
  q.ln_eps = p.ln_eps;
  const int64_t threads = (int64_t)p.M * q.cpr;
  hipLaunchKernelGGL(splitk_epilogue_kernel<E>, dim3((unsigned)((threads + 63) / 64)), dim3(64),
                     0, s, q);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(Epi epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if ((a.ccls != nullptr || epi == Epi::Patch) && a.tokens < 1) return hipErrorInvalidValue;
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
  p.patch_shift = -1;
  for (int sh = 0; sh < 16; ++sh)
    if (a.patch == (1 << sh)) p.patch_shift = sh;
  p.chans = a.chans;
  p.grid = a.grid;
  p.tokens = a.tokens;
  p.cls = a.cls;
  p.pos = a.pos;
  p.ldpos = a.ldpos > 0 ? a.ldpos : a.N;
  p.ccls = a.ccls;
  p.relu = a.relu ? 1 : 0;
  p.plan = a.plan;
  p.res = static_cast<const uint16_t*>(a.res);
  p.ldres = a.ldres;
  p.aux = static_cast<uint16_t*>(a.aux);
  p.ldaux = a.ldaux;
  p.ksplit = a.ksplit;
  p.kchunk = a.kchunk;
  p.c_split = a.c_split;
  p.ln_out = a.ln_out;
  p.ln_in = a.ln_in;
  p.ln_ld = a.ln_ld;
  p.ln_colsum = a.ln_colsum;
  p.ln_eps = a.ln_eps;
  const int64_t nseg_n = (a.N + 63) / 64, nseg_k = (a.K + 63) / 64;
  if (a.ln_out != nullptr && (epi != Epi::BiasResid && epi != Epi::Patch || a.N % 8 != 0 ||
                              a.ln_ld < nseg_n || a.ln_ld % 2 != 0))
    return hipErrorInvalidValue;
  if (a.ln_in != nullptr && (epi != Epi::Bias && epi != Epi::BiasGelu || a.ln_colsum == nullptr ||
                             a.ln_ld < nseg_k || a.ln_ld % 2 != 0 || !(a.ln_eps > 0.0f)))
    return hipErrorInvalidValue;
  if (a.ksplit > 1 && (epi != Epi::BiasF32 || a.kchunk < kBK || a.kchunk % kBK != 0 ||
                       (int64_t)(a.ksplit - 1) * a.kchunk >= a.K || a.c_split < (int64_t)a.M * a.ldc))
    return hipErrorInvalidValue;
  if (epi == Epi::GeluBwd && (a.aux == nullptr || a.ldaux < a.N || a.ldaux % 8 != 0))
    return hipErrorInvalidValue;
  if (a.res != nullptr && (a.ldres < a.N || a.ldres % 8 != 0)) return hipErrorInvalidValue;
  if (a.plan < 0 || a.plan >= kTilePlans) return hipErrorInvalidValue;
  if (a.aux != nullptr && epi == Epi::BiasGelu && (a.ldaux < a.N || a.ldaux % 8 != 0))
    return hipErrorInvalidValue;
  // Small M: split K over more workgroups when the caller gave a workspace,
  // in as many chunks as the planner's model chooses (plan 0) or as a split
  // plan forces (kSplitPlan0 and up); a forced tile plan never splits.
  const bool split_ok = a.ws != nullptr && a.ksplit <= 1 && !a.relu && a.aux == nullptr &&
                        p.bias != nullptr &&
                        (epi == Epi::Bias || epi == Epi::BiasGelu || epi == Epi::BiasResid);
  int ksplit = 1, kchunk = 0;
  if (a.plan >= kSplitPlan0) {
    if (!split_ok) return hipErrorNotSupported;
    ksplit = forced_split(p, a.ws_bytes, kSplitChunks[a.plan - kSplitPlan0], &kchunk);
    if (ksplit < 2) return hipErrorNotSupported;
  } else if (a.plan == 0 && split_ok) {
    ksplit = split_plan(p, a.ws_bytes, &kchunk);
  }
  if (ksplit > 1) {
    switch (epi) {
      case Epi::Bias: return launch_split<Epi::Bias>(p, a.ws, ksplit, kchunk, s);
      case Epi::BiasGelu: return launch_split<Epi::BiasGelu>(p, a.ws, ksplit, kchunk, s);
      default: return launch_split<Epi::BiasResid>(p, a.ws, ksplit, kchunk, s);
    }
  }
  switch (epi) {
    case Epi::Bias: return launch_epi<Epi::Bias>(p, s);
    case Epi::BiasGelu: return launch_epi<Epi::BiasGelu>(p, s);
    case Epi::BiasResid: return launch_epi<Epi::BiasResid>(p, s);
    case Epi::BiasF32: return launch_epi<Epi::BiasF32>(p, s);
    case Epi::Patch: return launch_epi<Epi::Patch>(p, s);
    case Epi::GeluBwd: return launch_epi<Epi::GeluBwd>(p, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_conv_bf16(const ConvArgs& a, hipStream_t s) {
  const int T = a.KH * a.KW;
  // Row-window form: each tap (kernel row) reads Ca consecutive elements from
  // its pixel on, i.e. a window of Ca / Cs pixels along the row.
  const bool win = a.row_window > 0;
  const int kw_out = win ? a.row_window : a.KW;
  if (a.batch < 0 || a.H < 1 || a.W < 1 || a.KH < 1 || a.KW < 1 || a.stride < 1 || a.pad < 0 ||
      a.N < 1 || a.Ca < 8 || (a.Ca & 7) != 0 || a.Cs < 1 || a.wseg < a.Ca || (a.wseg & 7) != 0 ||
      a.ldw < (int64_t)T * a.wseg || (a.ldw & 7) != 0 || a.ldc < a.N || (a.ldc & 7) != 0 ||
      T > 64 || a.plan < 0 || a.plan >= kTilePlans)
    return hipErrorInvalidValue;
  if (win ? (a.KW != 1 || a.pad != 0 || (a.Cs & 3) != 0 || (a.stride * a.Cs) % 8 != 0 ||
             (a.W * a.Cs) % 8 != 0 || a.Ca < a.row_window * a.Cs)
          : ((a.Cs & 7) != 0 || a.Ca > a.Cs))
    return hipErrorInvalidValue;
  const int Ho = (a.H + 2 * a.pad - a.KH) / a.stride + 1;
  const int Wo = (a.W + 2 * a.pad - kw_out) / a.stride + 1;
  if (Ho < 1 || Wo < 1) return hipErrorInvalidValue;
  if (a.batch == 0) return hipSuccess;
  const int64_t limit = ((int64_t)1 << 31) - 1;
  const int64_t w_bytes = ((int64_t)(a.N - 1) * a.ldw + (int64_t)T * a.wseg) * 2;
  const int64_t img_bytes = (int64_t)a.H * a.W * a.Cs * 2;
  if (w_bytes > limit || img_bytes > limit) return hipErrorInvalidValue;
  // K steps: Ca > 32 takes ceil(Ca / 64) steps per tap; otherwise taps
  // share a step, each spanning Cp = the next power of two >= Ca.
  // (Several taps a step need their pixel offsets, ((KH - 1) * W + KW - 1) *
  // Cs * 2 bytes at most, to fit 24 bits; otherwise one tap a step.)
  int tps = 1, cshift = 0;
  const int64_t max_tap_bytes = ((int64_t)(a.KH - 1) * a.W + (a.KW - 1)) * a.Cs * 2;
  if (a.Ca <= 32 && max_tap_bytes < (1 << 24) && (int64_t)a.W * a.Cs * 2 < (1 << 24)) {
    cshift = a.Ca <= 8 ? 3 : a.Ca <= 16 ? 4 : 5;
    tps = kBK >> cshift;
  }
  const int kwinv = 65536 / a.KW + 1;
  for (int t = 0; t < T + tps; ++t)  // the division by multiplication is exact here
    if ((t * kwinv) >> 16 != t / a.KW) return hipErrorInvalidValue;
  const int nc = (a.Ca + kBK - 1) / kBK, ncinv = 65536 / nc + 1;
  for (int kt = 0; kt <= T * nc; ++kt)
    if ((kt * ncinv) >> 16 != kt / nc) return hipErrorInvalidValue;
  // The range checks take 32-bit offsets: run the batch in runs of images
  // whose input stays below 2 GiB.
  const int per = (int)std::min<int64_t>(a.batch, limit / img_bytes);
  for (int b0 = 0; b0 < a.batch; b0 += per) {
    const int nb = std::min(per, a.batch - b0);
    Params p{};
    p.A = static_cast<const uint16_t*>(a.x) + (int64_t)b0 * a.H * a.W * a.Cs;
    p.W = static_cast<const uint16_t*>(a.weight);
    p.ldw = a.ldw;
    p.C = static_cast<uint16_t*>(a.C) + (int64_t)b0 * Ho * Wo * a.ldc;
    p.ldc = a.ldc;
    p.bias = a.bias;
    p.M = nb * Ho * Wo;
    p.N = a.N;
    p.K = T * a.Ca;
    p.relu = a.relu ? 1 : 0;
    p.plan = a.plan;
    p.cv_H = a.H; p.cv_W = a.W; p.cv_Cs = a.Cs; p.cv_Ca = a.Ca; p.cv_KW = a.KW; p.cv_T = T;
    p.cv_stride = a.stride; p.cv_pad = a.pad; p.cv_Ho = Ho; p.cv_Wo = Wo; p.cv_wseg = (int)a.wseg;
    p.cv_nc = (a.Ca + kBK - 1) / kBK;
    p.cv_tps = tps; p.cv_cshift = cshift; p.cv_kwinv = kwinv; p.cv_ncinv = ncinv;
    p.cv_rowb = a.W * a.Cs * 2; p.cv_pixb = a.Cs * 2;
    p.a_bytes = (int)(nb * img_bytes);
    p.w_bytes = (int)w_bytes;
    const hipError_t e = launch_epi<Epi::Bias, true>(p, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace elasto
