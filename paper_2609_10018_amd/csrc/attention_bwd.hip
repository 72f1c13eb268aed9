// Backward of the multi-head self-attention (Eq. 3) over the active head
// slots, bf16 with head_dim 64, fp32 accumulation, for the growth step.
//
// With S = q k^T * scale, P = softmax(S), o = P v and the incoming gradient
// do, the gradients are dv = P^T do, dS = P (.) (dP - rowsum(dP (.) P)) * scale
// with dP = do v^T, dq = dS k and dk = dS^T q.  Two kernels, one workgroup of
// 8 waves per (sequence, head slot):
//
// * dq kernel (16-query blocks, one block per wave in turn): K and V are
//   staged whole in LDS (rows of 128 B, XOR-swizzled 16-byte chunks) and K
//   transposed (K^T, one row per feature).  S^T = K Q^T and dP^T = V dO^T
//   come from v_mfma_f32_16x16x32_bf16 exactly as in the forward kernel
//   (lane l holds query l%16 against keys 16j + 4*(l/16) + {0..3}), so the
//   softmax is exact in registers.  dS is fed back as the A operand of
//   dq = dS K with the 8 keys a lane holds for two key tiles as its k-slots,
//   K^T read with the same key-to-slot assignment.  The kernel also writes,
//   per query, the log2-domain log-sum-exp of the scaled scores and
//   rowsum(dP (.) P) for the second kernel.
// * dk/dv kernel (16-key blocks): Q and dO are staged in LDS as rows and
//   transposed.  S = Q K^T and dP = dO V^T are computed per 16x16 block with
//   the key on the lane (lane l holds queries 4*(l/16) + {0..3} of the block
//   against key l%16), P is rebuilt from the stored log-sum-exp, and the 8
//   queries a lane holds for two query tiles are the k-slots of
//   dv += P^T dO and dk += dS^T Q, whose B operands come from dO^T and Q^T.
//
// Padding rows (tokens past the last) re-read the last token; their
// probabilities are zero, so they add nothing, and their outputs are not
// stored.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;

constexpr int kHd = 64;
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kOs = 72;                // output staging row stride (elements)
constexpr int kOStage = 16 * kOs * 2;  // bytes per wave

__device__ __forceinline__ int k_off(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }

struct AttnBwdP {
  const uint16_t* qkv;  // [B*T][qs]: slot s holds q, k, v at s*192 + {0, 64, 128}
  int64_t qs;
  const uint16_t* dout;  // [B*T][ds]: slot s at s*64
  int64_t ds;
  uint16_t* dqkv;  // same layout as qkv
  int64_t dqs;
  float* stats;    // [B][heads][T][2]: log2-domain lse, rowsum(dP . P)
  int T, heads;
  float scale, scale_log2;
};

// Stage rows [0, 16*NT) of a [T][64] bf16 operand (row stride ld) into LDS as
// swizzled 128-byte rows by direct loads; rows past T re-read row T-1.
template <int NT>
__device__ __forceinline__ void stage_rows(const uint16_t* src, int64_t ld, int T, char* dst,
                                           int wave, int lane) {
#pragma unroll
  for (int i = 0; i < (2 * NT + kWaves - 1) / kWaves; ++i) {
    const int blk = wave + kWaves * i;
    if (blk < 2 * NT) {
      const int r = blk * 8 + (lane >> 3);
      const int c = (lane & 7) ^ (r & 7);
      const uint16_t* g = src + (int64_t)min(r, T - 1) * ld + c * 8;
      __builtin_amdgcn_global_load_lds((global_void*)g, (lds_void*)(dst + blk * 1024), 16, 0, 0);
    }
  }
}

// Stage the transpose of the same operand: dst[c][r] (row stride VS), rows
// past T re-read row T-1.  All loads are issued before the LDS writes.
template <int NT, int VS>
__device__ __forceinline__ void stage_transposed(const uint16_t* src, int64_t ld, int T,
                                                 uint16_t* dst, int tid) {
  constexpr int TV = NT * 16;
  constexpr int kLoads = (TV * 8 + kThreads - 1) / kThreads;
  u32x4 vv[kLoads];
#pragma unroll
  for (int i = 0; i < kLoads; ++i) {
    const int idx = tid + kThreads * i, r = min(idx >> 3, T - 1), c = idx & 7;
    vv[i] = *reinterpret_cast<const u32x4*>(src + (int64_t)r * ld + c * 8);
  }
#pragma unroll
  for (int i = 0; i < kLoads; ++i) {
    const int idx = tid + kThreads * i, r = idx >> 3, c = idx & 7;
    if (r < TV) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        dst[(c * 8 + e) * VS + r] =
            (uint16_t)((e & 1) ? (vv[i][e >> 1] >> 16) : (vv[i][e >> 1] & 0xffffu));
    }
  }
}

// B operand of a 16x16x32 product over two 16-row tiles (2t, 2t+1) of an
// operand staged transposed (rows = features): 4 consecutive rows of each
// tile, as the k-slots a lane holds.
template <int VS>
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* tr, int feat, int t, int lg,
                                             bool has_hi) {
  const uint16_t* p = tr + feat * VS + t * 32 + 4 * lg;
  const u32x2 lo = *reinterpret_cast<const u32x2*>(p);
  u32x2 hi = {0u, 0u};
  if (has_hi) hi = *reinterpret_cast<const u32x2*>(p + 16);
  const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
  return __builtin_bit_cast(bf16x8, w);
}

// Write a wave's 16 x 64 fp32 tile (lane holds rows 4*lg + r, column
// n*16 + lq of acc[n][r]) as bf16 rows row0 + [0, 16) of dst (stride ld),
// skipping rows >= T; goes through the wave's LDS staging block.
__device__ __forceinline__ void store_tile(const f32x4* acc, uint16_t* ost, uint16_t* dst,
                                           int64_t ld, int row0, int T, int lane) {
  const int lq = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int n = 0; n < 4; ++n) ost[(4 * lg + r) * kOs + n * 16 + lq] = f32_to_bf16(acc[n][r]);
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14));  // LDS writes done
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int rr = h * 8 + (lane >> 3), c = lane & 7;
    const u32x4 w = *reinterpret_cast<const u32x4*>(ost + rr * kOs + c * 8);
    if (row0 + rr < T) *reinterpret_cast<u32x4*>(dst + (int64_t)(row0 + rr) * ld + c * 8) = w;
  }
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14));  // reads done before reuse
}

template <int NT>
__global__ __launch_bounds__(kThreads, 1) void attn_bwd_dq_kernel(AttnBwdP p) {
  constexpr int TV = NT * 16;
  constexpr int VS = TV + 4;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* kl = smem;
  char* vl = smem + NT * 2048;
  uint16_t* kt = reinterpret_cast<uint16_t*>(smem + 2 * NT * 2048);
  uint16_t* ost = reinterpret_cast<uint16_t*>(smem + 2 * NT * 2048 + kHd * VS * 2);

  const int T = p.T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x / p.heads, s = blockIdx.x - b * p.heads;
  const uint16_t* base = p.qkv + (int64_t)b * T * p.qs + (int64_t)s * 3 * kHd;
  const uint16_t* dbase = p.dout + (int64_t)b * T * p.ds + (int64_t)s * kHd;
  const int lq = lane & 15, lg = lane >> 4;

  stage_rows<NT>(base + kHd, p.qs, T, kl, wave, lane);
  stage_rows<NT>(base + 2 * kHd, p.qs, T, vl, wave, lane);
  stage_transposed<NT, VS>(base + kHd, p.qs, T, kt, tid);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const float c2 = p.scale_log2;
  uint16_t* my_ost = ost + wave * (kOStage / 2);
  for (int qb = wave; qb < NT; qb += kWaves) {
    const int q0 = qb * 16;
    const int qrow = min(q0 + lq, T - 1);
    bf16x8 qf[2], df[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      qf[kk] = *reinterpret_cast<const bf16x8*>(base + (int64_t)qrow * p.qs + kk * 32 + lg * 8);
      df[kk] = *reinterpret_cast<const bf16x8*>(dbase + (int64_t)qrow * p.ds + kk * 32 + lg * 8);
    }
    f32x4 st[NT], dp[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(kl + k_off(j * 16 + lq, kk * 4 + lg));
        const bf16x8 va = *reinterpret_cast<const bf16x8*>(vl + k_off(j * 16 + lq, kk * 4 + lg));
        a0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[kk], a0, 0, 0, 0);
        a1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, df[kk], a1, 0, 0, 0);
      }
      st[j] = a0;
      dp[j] = a1;
      if ((j & 3) == 3) __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_sched_barrier(0);
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
    const float inv = 1.0f / sum;
    float dsum = 0.f;  // rowsum(dP . P) of query lq
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        st[j][r] *= inv;
        dsum = fmaf(st[j][r], dp[j][r], dsum);
      }
    dsum += __shfl_xor(dsum, 16, 64);
    dsum += __shfl_xor(dsum, 32, 64);
    if (lg == 0 && q0 + lq < T) {
      float* sp = p.stats + (((int64_t)b * p.heads + s) * T + q0 + lq) * 2;
      sp[0] = fmaf(mx, c2, log2f(sum));
      sp[1] = dsum;
    }
    __builtin_amdgcn_sched_barrier(0);

    f32x4 dq[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) dq[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < (NT + 1) / 2; ++kb) {
      const bool has_hi = 2 * kb + 1 < NT;
      const int hi_t = has_hi ? 2 * kb + 1 : 2 * kb;
      bf16x8 sa;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sa[r] = static_cast<__bf16>(st[2 * kb][r] * (dp[2 * kb][r] - dsum) * p.scale);
        sa[4 + r] = has_hi ? static_cast<__bf16>(st[hi_t][r] * (dp[hi_t][r] - dsum) * p.scale)
                           : static_cast<__bf16>(0.f);
      }
#pragma unroll
      for (int n = 0; n < 4; ++n)
        dq[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            sa, tr_operand<VS>(kt, n * 16 + lq, kb, lg, has_hi), dq[n], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    store_tile(dq, my_ost, p.dqkv + (int64_t)b * T * p.dqs + (int64_t)s * 3 * kHd, p.dqs, q0, T,
               lane);
  }
}

template <int NT>
__global__ __launch_bounds__(kThreads, 1) void attn_bwd_dkv_kernel(AttnBwdP p) {
  constexpr int TV = NT * 16;
  constexpr int VS = TV + 4;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* ql = smem;
  char* dl = smem + NT * 2048;
  uint16_t* qt = reinterpret_cast<uint16_t*>(smem + 2 * NT * 2048);
  uint16_t* dt = qt + kHd * VS;
  float* lse = reinterpret_cast<float*>(smem + 2 * NT * 2048 + 2 * kHd * VS * 2);
  float* dsm = lse + TV;
  uint16_t* ost = reinterpret_cast<uint16_t*>(dsm + TV);

  const int T = p.T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x / p.heads, s = blockIdx.x - b * p.heads;
  const uint16_t* base = p.qkv + (int64_t)b * T * p.qs + (int64_t)s * 3 * kHd;
  const uint16_t* dbase = p.dout + (int64_t)b * T * p.ds + (int64_t)s * kHd;
  const int lq = lane & 15, lg = lane >> 4;

  stage_rows<NT>(base, p.qs, T, ql, wave, lane);
  stage_rows<NT>(dbase, p.ds, T, dl, wave, lane);
  stage_transposed<NT, VS>(base, p.qs, T, qt, tid);
  stage_transposed<NT, VS>(dbase, p.ds, T, dt, tid);
  const float* sp = p.stats + ((int64_t)b * p.heads + s) * T * 2;
  for (int i = tid; i < TV; i += kThreads) {
    lse[i] = i < T ? sp[2 * i] : 0.f;
    dsm[i] = i < T ? sp[2 * i + 1] : 0.f;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const float c2 = p.scale_log2;
  uint16_t* my_ost = ost + wave * (kOStage / 2);
  uint16_t* obase = p.dqkv + (int64_t)b * T * p.dqs + (int64_t)s * 3 * kHd;
  for (int kb = wave; kb < NT; kb += kWaves) {
    const int key = min(kb * 16 + lq, T - 1);
    bf16x8 kf[2], vf[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      kf[kk] = *reinterpret_cast<const bf16x8*>(base + (int64_t)key * p.qs + kHd + kk * 32 + lg * 8);
      vf[kk] =
          *reinterpret_cast<const bf16x8*>(base + (int64_t)key * p.qs + 2 * kHd + kk * 32 + lg * 8);
    }
    f32x4 dk[4], dv[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) dk[n] = dv[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int qp = 0; qp < (NT + 1) / 2; ++qp) {
      bf16x8 pa, sa;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int qj = 2 * qp + t;
        if (qj < NT) {
          f32x4 sv = {0.f, 0.f, 0.f, 0.f}, dpv = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            const bf16x8 qa = *reinterpret_cast<const bf16x8*>(ql + k_off(qj * 16 + lq, kk * 4 + lg));
            const bf16x8 da = *reinterpret_cast<const bf16x8*>(dl + k_off(qj * 16 + lq, kk * 4 + lg));
            sv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, kf[kk], sv, 0, 0, 0);
            dpv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(da, vf[kk], dpv, 0, 0, 0);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int q = qj * 16 + 4 * lg + r;
            const float pv = q < T ? __builtin_amdgcn_exp2f(fmaf(sv[r], c2, -lse[q])) : 0.f;
            pa[4 * t + r] = static_cast<__bf16>(pv);
            sa[4 * t + r] = static_cast<__bf16>(pv * (dpv[r] - dsm[q]) * p.scale);
          }
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            pa[4 * t + r] = static_cast<__bf16>(0.f);
            sa[4 * t + r] = static_cast<__bf16>(0.f);
          }
        }
      }
      const bool has_hi = 2 * qp + 1 < NT;
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        dv[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            pa, tr_operand<VS>(dt, n * 16 + lq, qp, lg, has_hi), dv[n], 0, 0, 0);
        dk[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            sa, tr_operand<VS>(qt, n * 16 + lq, qp, lg, has_hi), dk[n], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    store_tile(dk, my_ost, obase + kHd, p.dqs, kb * 16, T, lane);
    store_tile(dv, my_ost, obase + 2 * kHd, p.dqs, kb * 16, T, lane);
  }
}

template <int NT>
hipError_t launch_bwd_nt(const AttnBwdP& p, int batch, hipStream_t s) {
  constexpr int VS = NT * 16 + 4;
  const size_t lds_dq = (size_t)2 * NT * 2048 + (size_t)kHd * VS * 2 + (size_t)kWaves * kOStage;
  const size_t lds_dkv = (size_t)2 * NT * 2048 + (size_t)2 * kHd * VS * 2 +
                         (size_t)2 * NT * 16 * 4 + (size_t)kWaves * kOStage;
  const unsigned grid = (unsigned)(batch * p.heads);
  hipLaunchKernelGGL(attn_bwd_dq_kernel<NT>, dim3(grid), dim3(kThreads), lds_dq, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_bwd_dkv_kernel<NT>, dim3(grid), dim3(kThreads), lds_dkv, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_bwd_bf16(const AttnBwdArgs& a, hipStream_t s) {
  if (a.batch <= 0 || a.heads <= 0 || a.tokens <= 0) return hipSuccess;
  if (a.head_dim != kHd || a.tokens > kAttnMaxTokens) return hipErrorInvalidValue;
  AttnBwdP p;
  p.qkv = static_cast<const uint16_t*>(a.qkv);
  p.qs = a.qkv_stride;
  p.dout = static_cast<const uint16_t*>(a.dout);
  p.ds = a.dout_stride;
  p.dqkv = static_cast<uint16_t*>(a.dqkv);
  p.dqs = a.dqkv_stride;
  p.stats = a.stats;
  p.T = a.tokens;
  p.heads = a.heads;
  p.scale = a.scale;
  p.scale_log2 = a.scale * 1.4426950408889634f;
  switch ((a.tokens + 15) / 16) {
    case 1: return launch_bwd_nt<1>(p, a.batch, s);
    case 2: return launch_bwd_nt<2>(p, a.batch, s);
    case 3: return launch_bwd_nt<3>(p, a.batch, s);
    case 4: return launch_bwd_nt<4>(p, a.batch, s);
    case 5: return launch_bwd_nt<5>(p, a.batch, s);
    case 6: return launch_bwd_nt<6>(p, a.batch, s);
    case 7: return launch_bwd_nt<7>(p, a.batch, s);
    case 8: return launch_bwd_nt<8>(p, a.batch, s);
    case 9: return launch_bwd_nt<9>(p, a.batch, s);
    case 10: return launch_bwd_nt<10>(p, a.batch, s);
    case 11: return launch_bwd_nt<11>(p, a.batch, s);
    case 12: return launch_bwd_nt<12>(p, a.batch, s);
    case 13: return launch_bwd_nt<13>(p, a.batch, s);
    case 14: return launch_bwd_nt<14>(p, a.batch, s);
    case 15: return launch_bwd_nt<15>(p, a.batch, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace elasto
