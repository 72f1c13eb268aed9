// Multi-head self-attention over the active heads (Eq. 3):
// o = softmax(q k^T * scale) v per (sequence, head slot).
//
// bf16 path (head_dim 64): one workgroup of 8 waves per (sequence, head
// slot), so no wave takes more than two of the (up to 15) query blocks (two
// workgroups, each with a share of the blocks, when the pairs are too few to
// fill the CUs: small batches).  K and
// V are staged whole in LDS by direct global->LDS loads, both in token-row
// layout (rows of 128 B, 16-byte chunks XOR-swizzled); padding keys past the
// last token repeat that token and are masked (zero probability).  Each wave
// takes 16-query blocks in turn and computes the score block transposed,
// S^T = K Q^T, with v_mfma_f32_16x16x32_bf16: lane l then holds the scores of
// query l%16 against keys 16j + 4*(l/16) + {0..3}.  The softmax of a query is
// reduced over its 4 lanes with two xor-shuffles and is exact (single pass:
// the whole key row fits in registers).  The probabilities are rounded to
// bf16 and are reused unchanged as the k-slots of the second product, which
// is also taken transposed, O^T = V^T P^T: the MFMA's k-slots are only
// labels, so the 8 keys a lane holds for two adjacent key tiles form its
// k-slots, and the V^T operand is read from the row-major V with the LDS
// transpose read (ds_read_b64_tr_b16: in each group of 16 lanes, lane i
// receives element i%4 of the 8-byte pieces that lanes i/4, 4 + i/4, 8 + i/4
// and 12 + i/4 address, so four key rows x 16 feature columns come back as
// four keys per lane, one column per lane).  Lane l then holds features
// 16n + 4*(l/16) + {0..3} of query l%16: the 1/rowsum normalisation is
// applied in fp32 and each lane writes 8-byte pieces of its query's row.
//
// fp32 path: a plain per-query loop (two passes over the keys: max, then
// exp-sum and weighted V sum), fp32 FMA throughout.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kHd = 64;
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kRsrcWord3 = 0x00020000;  // buffer resource: raw (unswizzled) 32-bit records

// Byte offset of logical 16-byte chunk c of token row r in a staged K or V.
__device__ __forceinline__ int kv_off(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }

struct AttnP {
  const uint16_t* qkv;
  int64_t qs;
  uint16_t* o;
  int64_t os;
  int T, heads;
  int parts;  // workgroups per (sequence, head slot), each a share of the query blocks
  float scale_log2;
};

// NT = ceil(T / 16) key tiles, fixed at compile time so that every loop over
// keys is fully unrolled and only the last tile carries the key < T mask.
template <int NT>
__global__ __launch_bounds__(kThreads, 2) void attention_bf16_kernel(AttnP p) {
  constexpr int KV = NT * 16 * 128;  // bytes of the staged K (and of V)
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int T = p.T;
  const char* kl = smem;
  const char* vl = smem + KV;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bs = blockIdx.x / p.parts, part = blockIdx.x - bs * p.parts;
  const int b = bs / p.heads, s = bs - b * p.heads;
  // Query blocks of this workgroup: part * 8 + wave, then every 8 * parts.
  const int qb0 = part * kWaves + wave, qstep = kWaves * p.parts;
  const uint16_t* base = p.qkv + (int64_t)b * T * p.qs + (int64_t)s * 3 * kHd;

  const int lq = lane & 15, lg = lane >> 4;
  // Q fragments of a 16-query block (B operand of S^T = K Q^T); rows past the
  // last token re-read token T-1 and their outputs are dropped.
  auto load_q = [&](int qb, bf16x8* qf) {
    const int q = min(qb * 16 + lq, T - 1);
    const uint16_t* qp = base + (int64_t)q * p.qs + lg * 8;
    qf[0] = *reinterpret_cast<const bf16x8*>(qp);
    qf[1] = *reinterpret_cast<const bf16x8*>(qp + 32);
  };
  bf16x8 qf[2];
  if (qb0 < NT) load_q(qb0, qf);

  // K and V: direct global->LDS loads in 1-KB blocks of 8 token rows (blocks
  // 0 .. 2NT-1 are K, the next 2NT are V).  Lane l lands at block + 16 l,
  // i.e. row 8*blk + l/8, physical chunk l%8, so it fetches the logical chunk
  // that kv_off() places there.  Rows past the last token re-read token T-1:
  // their scores are masked out and their probabilities are 0.  Each wave
  // issues its K blocks first, then as many V blocks (wave + 8i < 2NT for
  // both), so the first scores are computed while V is still arriving.
  constexpr int kLoadIters = (2 * NT + kWaves - 1) / kWaves;
#pragma unroll
  for (int isv = 0; isv < 2; ++isv)
#pragma unroll
    for (int i = 0; i < kLoadIters; ++i) {
      const int rb = wave + kWaves * i;  // block of 8 rows within K or V
      if (rb < 2 * NT) {
        const int r = rb * 8 + (lane >> 3);
        const int c = (lane & 7) ^ (r & 7);
        const uint16_t* src = base + (int64_t)min(r, T - 1) * p.qs + (1 + isv) * kHd + c * 8;
        __builtin_amdgcn_global_load_lds((global_void*)src,
                                         (lds_void*)(smem + (isv * 2 * NT + rb) * 1024), 16, 0, 0);
      }
    }
  // Nothing reads the staged rows by register dependence.  K: wait until at
  // most this wave's V loads are in flight (loads complete in issue order for
  // the counter; the Q loads came first), then for every wave.
  const int nkv = wave < 2 * NT ? (2 * NT - 1 - wave) / kWaves + 1 : 0;
  static_assert(kLoadIters <= 4, "K/V loads per wave exceed the wait cases");
  switch (nkv) {
    case 0: __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xF << 8)); break;
    case 1: __builtin_amdgcn_s_waitcnt(1 | (0x7 << 4) | (0xF << 8)); break;
    case 2: __builtin_amdgcn_s_waitcnt(2 | (0x7 << 4) | (0xF << 8)); break;
    case 3: __builtin_amdgcn_s_waitcnt(3 | (0x7 << 4) | (0xF << 8)); break;
    default: __builtin_amdgcn_s_waitcnt(4 | (0x7 << 4) | (0xF << 8)); break;
  }
  __syncthreads();

  // Output rows of this (sequence, head slot): T rows of p.os elements from
  // column s*64; an offset of nrec drops the store (rows past the last token).
  const int nrec = T * (int)p.os * 2;
  const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
      p.o + (int64_t)b * T * p.os + (int64_t)s * kHd, (short)0, nrec, kRsrcWord3);
  const float c2 = p.scale_log2;
  for (int qb = qb0; qb < NT; qb += qstep) {
    const int q0 = qb * 16;
    f32x4 st[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(kl + kv_off(j * 16 + lq, kk * 4 + lg));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[kk], acc, 0, 0, 0);
      }
      st[j] = acc;
      // Bound how far the scheduler hoists LDS reads (register pressure).
      if ((j & 3) == 3) __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_sched_barrier(0);
    bf16x8 qn[2];
    if (qb + qstep < NT) load_q(qb + qstep, qn);
    // Keys of the last tile at or past T do not exist.
    bool valid[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) valid[r] = (NT - 1) * 16 + 4 * lg + r < T;
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        mx = fmaxf(mx, (j < NT - 1 || valid[r]) ? st[j][r] : -INFINITY);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float off = -mx * c2;
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float e = __builtin_amdgcn_exp2f(fmaf(st[j][r], c2, off));
        if (j == NT - 1) e = valid[r] ? e : 0.f;
        st[j][r] = e;
        sum += e;
      }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    __builtin_amdgcn_sched_barrier(0);
    // V: before the first product with it, every V load of every wave.  Each
    // wave passes this barrier once (here on its first block, or after the
    // loop when it has none).
    if (qb == qb0) {
      __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
      __syncthreads();
    }

    // O^T = V^T P^T over key pairs of tiles (2kb, 2kb+1): k-slot 8*lg + r is
    // key 32kb + 4lg + r, k-slot 8*lg + 4 + r is key 32kb + 16 + 4lg + r.
    f32x4 o[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) o[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int vr = 4 * lg + (lq >> 2);  // key row this lane addresses, within a 32-key pair
#pragma unroll
    for (int kb = 0; kb < (NT + 1) / 2; ++kb) {
      const bool has_hi = 2 * kb + 1 < NT;
      bf16x8 pa;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pa[r] = static_cast<__bf16>(st[2 * kb][r]);
        pa[4 + r] = has_hi ? static_cast<__bf16>(st[has_hi ? 2 * kb + 1 : 2 * kb][r])
                           : static_cast<__bf16>(0.f);
      }
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        // This lane addresses columns 16n + 4(lq%4) .. +3 of key row 32kb + vr
        // (and of the row 16 keys further for the upper k-slots).
        const int col = n * 16 + 4 * (lq & 3), half = (col & 4) * 2;
        const int r0 = kb * 32 + vr;
        const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4*)(vl + kv_off(r0, col >> 3) + half)));
        u32x2 hi = {0u, 0u};
        if (has_hi)
          hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4*)(vl + kv_off(r0 + 16, col >> 3) + half)));
        const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
        o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w), pa, o[n],
                                                       0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // Lane (lg, lq) holds O[q0 + lq][16n + 4lg + r], r = 0..3.
    const float inv = 1.0f / sum;  // for query lq
    const int q = q0 + lq;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const u32x2 w = {pack_bf16x2(o[n][0] * inv, o[n][1] * inv),
                       pack_bf16x2(o[n][2] * inv, o[n][3] * inv)};
      __builtin_amdgcn_raw_buffer_store_b64(w, ro, q < T ? (q * (int)p.os + 16 * n + 4 * lg) * 2 : nrec,
                                            0, 0);
    }
    qf[0] = qn[0];
    qf[1] = qn[1];
  }
  if (qb0 >= NT) {
    __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
    __syncthreads();
  }
}

template <int NT>
hipError_t launch_attn_nt(AttnP p, int batch, int heads, hipStream_t s) {
  const size_t lds = 2 * (size_t)NT * 16 * 128;
  // Few (sequence, head slot) pairs (small batches, narrow modes): split each
  // one's query blocks over more workgroups (each stages K and V itself), so
  // that more CUs work and a wave takes one block instead of two.
  constexpr int kCUs = 256;
  const int pairs = batch * heads;
  p.parts = std::max(1, std::min((NT + kWaves - 1) / kWaves, kCUs / std::max(pairs, 1)));
  hipLaunchKernelGGL(attention_bf16_kernel<NT>, dim3((unsigned)(pairs * p.parts)), dim3(kThreads),
                     lds, s, p);
  return hipGetLastError();
}

struct AttnF {
  const float* qkv;
  int64_t qs;
  float* o;
  int64_t os;
  int T, heads, hd;
  float scale;
};

constexpr int kHdMaxF32 = 128;

__global__ __launch_bounds__(256) void attention_f32_kernel(AttnF p) {
  const int b = blockIdx.x / p.heads, s = blockIdx.x - b * p.heads;
  const int hd = p.hd;
  const float* base = p.qkv + (int64_t)b * p.T * p.qs + (int64_t)s * 3 * hd;
  for (int q = threadIdx.x; q < p.T; q += blockDim.x) {
    float qv[kHdMaxF32];
    const float* qp = base + (int64_t)q * p.qs;
    for (int c = 0; c < hd; ++c) qv[c] = qp[c];
    float mx = -INFINITY;
    for (int j = 0; j < p.T; ++j) {
      const float* kp = base + (int64_t)j * p.qs + hd;
      float dot = 0.f;
      for (int c = 0; c < hd; ++c) dot = fmaf(qv[c], kp[c], dot);
      mx = fmaxf(mx, dot * p.scale);
    }
    float acc[kHdMaxF32];
    for (int c = 0; c < hd; ++c) acc[c] = 0.f;
    float sum = 0.f;
    for (int j = 0; j < p.T; ++j) {
      const float* kp = base + (int64_t)j * p.qs + hd;
      const float* vp = kp + hd;
      float dot = 0.f;
      for (int c = 0; c < hd; ++c) dot = fmaf(qv[c], kp[c], dot);
      const float e = expf(dot * p.scale - mx);
      sum += e;
      for (int c = 0; c < hd; ++c) acc[c] = fmaf(e, vp[c], acc[c]);
    }
    const float inv = 1.0f / sum;
    float* op = p.o + ((int64_t)b * p.T + q) * p.os + (int64_t)s * hd;
    for (int c = 0; c < hd; ++c) op[c] = acc[c] * inv;
  }
}

}  // namespace

hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.batch <= 0 || a.heads <= 0 || a.tokens <= 0) return hipSuccess;
  if (a.head_dim != kHd || a.tokens > kAttnMaxTokens) return hipErrorInvalidValue;
  // The output of a (sequence, head slot) is addressed as one buffer range of
  // T rows: the rows must hold every head slot and the range must fit 31 bits.
  if (a.o_stride < (int64_t)a.heads * kHd || a.qkv_stride < (int64_t)a.heads * 3 * kHd ||
      (int64_t)a.tokens * a.o_stride * 2 > INT32_MAX)
    return hipErrorInvalidValue;
  AttnP p;
  p.qkv = static_cast<const uint16_t*>(a.qkv);
  p.qs = a.qkv_stride;
  p.o = static_cast<uint16_t*>(a.o);
  p.os = a.o_stride;
  p.T = a.tokens;
  p.heads = a.heads;
  p.scale_log2 = a.scale * 1.4426950408889634f;
  switch ((a.tokens + 15) / 16) {
    case 1: return launch_attn_nt<1>(p, a.batch, a.heads, s);
    case 2: return launch_attn_nt<2>(p, a.batch, a.heads, s);
    case 3: return launch_attn_nt<3>(p, a.batch, a.heads, s);
    case 4: return launch_attn_nt<4>(p, a.batch, a.heads, s);
    case 5: return launch_attn_nt<5>(p, a.batch, a.heads, s);
    case 6: return launch_attn_nt<6>(p, a.batch, a.heads, s);
    case 7: return launch_attn_nt<7>(p, a.batch, a.heads, s);
    case 8: return launch_attn_nt<8>(p, a.batch, a.heads, s);
    case 9: return launch_attn_nt<9>(p, a.batch, a.heads, s);
    case 10: return launch_attn_nt<10>(p, a.batch, a.heads, s);
    case 11: return launch_attn_nt<11>(p, a.batch, a.heads, s);
    case 12: return launch_attn_nt<12>(p, a.batch, a.heads, s);
    case 13: return launch_attn_nt<13>(p, a.batch, a.heads, s);
    case 14: return launch_attn_nt<14>(p, a.batch, a.heads, s);
    case 15: return launch_attn_nt<15>(p, a.batch, a.heads, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention_f32(const AttnArgs& a, hipStream_t s) {
  if (a.batch <= 0 || a.heads <= 0 || a.tokens <= 0) return hipSuccess;
  if (a.head_dim > kHdMaxF32 || a.head_dim <= 0) return hipErrorInvalidValue;
  AttnF p;
  p.qkv = static_cast<const float*>(a.qkv);
  p.qs = a.qkv_stride;
  p.o = static_cast<float*>(a.o);
  p.os = a.o_stride;
  p.T = a.tokens;
  p.heads = a.heads;
  p.hd = a.head_dim;
  p.scale = a.scale;
  hipLaunchKernelGGL(attention_f32_kernel, dim3((unsigned)(a.batch * a.heads)), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace elasto
