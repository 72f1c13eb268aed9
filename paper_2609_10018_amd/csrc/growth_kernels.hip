// Elementwise, reduction and data-movement kernels of the growth step
// (Section 4.2): the backward's transposes and LayerNorm backward, the
// cross-entropy loss, bias gradients, split-K reduction, the selective
// clipping norm (Eq. 9's G is applied by computing gradients only for the
// re-introduced slices), and the masked update with fp32 master weights.
#include "common.h"
#include "kernels.h"

namespace elasto {
namespace {

inline unsigned grid_for(int64_t n, int block) { return (unsigned)((n + block - 1) / block); }

// ------------------------------------------------------------- transpose
// out[c][r] = in[r][c0 + c] for r < R, c < n.  64x64 tiles through LDS; any
// alignment of c0 (elementwise loads, coalesced along the row).
constexpr int kTT = 64;
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ in,
                                                        int64_t ldi, int64_t c0, int R, int n,
                                                        uint16_t* __restrict__ out, int64_t ldo) {
  __shared__ uint16_t tile[kTT][kTT + 2];
  const int r0 = blockIdx.y * kTT, cb = blockIdx.x * kTT;
  const int t = threadIdx.x;
  {
    const int c = t & 63, rs = (t >> 6) * 16;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int r = r0 + rs + e;
      tile[rs + e][c] = (r < R && cb + c < n) ? in[(int64_t)r * ldi + c0 + cb + c] : (uint16_t)0;
    }
  }
  __syncthreads();
  const int oc = t >> 2, seg = (t & 3) * 16;  // output row cb + oc, input rows r0 + seg + [0, 16)
  if (cb + oc >= n) return;
  uint16_t* op = out + (int64_t)(cb + oc) * ldo + r0 + seg;
  if (r0 + seg + 16 <= R) {
    u32x4 w0, w1;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      w0[h] = (uint32_t)tile[seg + 2 * h][oc] | ((uint32_t)tile[seg + 2 * h + 1][oc] << 16);
      w1[h] = (uint32_t)tile[seg + 8 + 2 * h][oc] | ((uint32_t)tile[seg + 9 + 2 * h][oc] << 16);
    }
    *reinterpret_cast<u32x4*>(op) = w0;
    *reinterpret_cast<u32x4*>(op + 8) = w1;
  } else {
    for (int e = 0; e < 16 && r0 + seg + e < R; ++e) op[e] = tile[seg + e][oc];
  }
}

// --------------------------------------------------------- LayerNorm bwd
// One wave per row: xhat = (x - mean) * rstd recomputed from x (bf16),
// g = dy * gamma, dx = rstd * (g - mean(g) - xhat * mean(g * xhat));
// dX[row] += dx (fp32) and dXb[row] = bf16(dX[row]).
constexpr int kLnMaxPerLane = 32;  // d <= 2048
__global__ __launch_bounds__(256) void layernorm_bwd_kernel(
    const uint16_t* __restrict__ x, int64_t ldx, const uint16_t* __restrict__ dy, int64_t ldy,
    const float* __restrict__ gamma, float eps, int rows, int d, float* __restrict__ dX,
    int64_t lddx, uint16_t* __restrict__ dXb, int64_t lddxb) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + wave;
  if (row >= rows) return;
  const uint16_t* xr = x + (int64_t)row * ldx;
  const uint16_t* gr = dy + (int64_t)row * ldy;
  float xv[kLnMaxPerLane], gv[kLnMaxPerLane];
  float s = 0.f;
  int cnt = 0;
#pragma unroll
  for (int i = 0; i < kLnMaxPerLane; ++i) {
    const int c = lane + 64 * i;
    xv[i] = c < d ? bf16_to_f32(xr[c]) : 0.f;
    s += xv[i];
    cnt += c < d;
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  const float mean = s / (float)d;
  float v = 0.f;
#pragma unroll
  for (int i = 0; i < kLnMaxPerLane; ++i) {
    const int c = lane + 64 * i;
    const float dd = c < d ? xv[i] - mean : 0.f;
    v = fmaf(dd, dd, v);
  }
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const float rstd = 1.0f / sqrtf(v / (float)d + eps);
  float sg = 0.f, sgx = 0.f;
#pragma unroll
  for (int i = 0; i < kLnMaxPerLane; ++i) {
    const int c = lane + 64 * i;
    if (c < d) {
      xv[i] = (xv[i] - mean) * rstd;
      gv[i] = bf16_to_f32(gr[c]) * gamma[c];
      sg += gv[i];
      sgx = fmaf(gv[i], xv[i], sgx);
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    sg += __shfl_xor(sg, o, 64);
    sgx += __shfl_xor(sgx, o, 64);
  }
  sg /= (float)d;
  sgx /= (float)d;
  float* dxr = dX + (int64_t)row * lddx;
  uint16_t* dbr = dXb + (int64_t)row * lddxb;
#pragma unroll
  for (int i = 0; i < kLnMaxPerLane; ++i) {
    const int c = lane + 64 * i;
    if (c < d) {
      const float nv = dxr[c] + rstd * (gv[i] - sg - xv[i] * sgx);
      dxr[c] = nv;
      dbr[c] = f32_to_bf16(nv);
    }
  }
  (void)cnt;
}

// ---------------------------------------------------------- cross-entropy
// One workgroup per image: loss_b = log sum exp(z) - z[label];
// dlogits = (softmax(z) - onehot(label)) / batch, bf16.  A label outside
// [0, C) gives a NaN loss and no one-hot term.
__global__ __launch_bounds__(256) void cross_entropy_kernel(const float* __restrict__ logits,
                                                            int64_t ldl,
                                                            const int32_t* __restrict__ labels,
                                                            int C, int batch,
                                                            uint16_t* __restrict__ dlogits,
                                                            int64_t ldd,
                                                            float* __restrict__ rowloss) {
  __shared__ float red[8];
  const int b = blockIdx.x, t = threadIdx.x;
  const float* z = logits + (int64_t)b * ldl;
  float mx = -INFINITY;
  for (int c = t; c < C; c += 256) mx = fmaxf(mx, z[c]);
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  if ((t & 63) == 0) red[t >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float s = 0.f;
  for (int c = t; c < C; c += 256) s += expf(z[c] - mx);
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((t & 63) == 0) red[4 + (t >> 6)] = s;
  __syncthreads();
  s = (red[4] + red[5]) + (red[6] + red[7]);
  const int y = labels[b];
  const bool ok = y >= 0 && y < C;
  const float inv = 1.0f / s, ib = 1.0f / (float)batch;
  for (int c = t; c < C; c += 256) {
    const float pr = expf(z[c] - mx) * inv;
    dlogits[(int64_t)b * ldd + c] = f32_to_bf16((pr - (ok && c == y ? 1.0f : 0.0f)) * ib);
  }
  if (t == 0) rowloss[b] = ok ? logf(s) + mx - z[y] : NAN;
}

// --------------------------------------------------------- small reductions
// out[r] = sum_{c < n} in[r][c] (bf16 in, fp32 sum), one wave per row.
__global__ __launch_bounds__(256) void rowsum_kernel(const uint16_t* __restrict__ in, int64_t ld,
                                                     int rows, int n, float* __restrict__ out) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave;
  if (r >= rows) return;
  const uint16_t* p = in + (int64_t)r * ld;
  float s = 0.f;
  for (int c = lane; c < n; c += 64) s += bf16_to_f32(p[c]);
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) out[r] = s;
}

// out[r][c] = sum_s part[s][r][c] (fp32), part chunks c_split apart,
// partial rows of ldp elements, out rows of ldo.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            int64_t c_split, int ksplit, int rows,
                                                            int cols, int64_t ldp,
                                                            float* __restrict__ out, int64_t ldo) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (int64_t)rows * cols) return;
  const int r = (int)(id / cols), c = (int)(id - (int64_t)r * cols);
  float s = 0.f;
  for (int k = 0; k < ksplit; ++k) s += part[k * c_split + (int64_t)r * ldp + c];
  out[(int64_t)r * ldo + c] = s;
}

// Sum of squares of a fp32 array: one partial per workgroup.
constexpr int kSqBlocks = 1024;
__global__ __launch_bounds__(256) void sumsq_kernel(const float* __restrict__ g, int64_t n,
                                                    float* __restrict__ part) {
  __shared__ float red[4];
  float s = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    s = fmaf(g[i], g[i], s);
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// stats = {mean loss, |G . grad|, clip factor}; the factor is also what the
// update kernel reads.
__global__ __launch_bounds__(256) void growth_finish_kernel(const float* __restrict__ part,
                                                            int nparts,
                                                            const float* __restrict__ rowloss,
                                                            int batch, float clip,
                                                            float* __restrict__ stats) {
  __shared__ float red[8];
  float s = 0.f, l = 0.f;
  for (int i = threadIdx.x; i < nparts; i += 256) s += part[i];
  for (int i = threadIdx.x; i < batch; i += 256) l += rowloss[i];
  for (int o = 32; o > 0; o >>= 1) {
    s += __shfl_xor(s, o, 64);
    l += __shfl_xor(l, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = s;
    red[4 + (threadIdx.x >> 6)] = l;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const float norm = sqrtf((red[0] + red[1]) + (red[2] + red[3]));
    stats[0] = ((red[4] + red[5]) + (red[6] + red[7])) / (float)batch;
    stats[1] = norm;
    stats[2] = norm > clip ? clip / norm : 1.0f;
  }
}

// ----------------------------------------------------------------- update
// One workgroup row per slice (blockIdx.y), elements strided over blockIdx.x.
__global__ __launch_bounds__(256) void growth_update_kernel(const GrowthSlice* __restrict__ sl,
                                                            const float* __restrict__ grad,
                                                            float* __restrict__ master,
                                                            uint8_t* __restrict__ packed,
                                                            const float* __restrict__ stats,
                                                            float lr) {
  const GrowthSlice d = sl[blockIdx.y];
  const int64_t n = (int64_t)d.rows * d.cols;
  const float step = lr * stats[2];
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int r = (int)(i / d.cols), c = (int)(i - (int64_t)r * d.cols);
    const float g = grad[d.grad_off + (int64_t)r * d.grad_ld + c];
    const int64_t e = (int64_t)r * d.ld + c;
    if (d.is_bf16) {
      const int64_t idx = d.packed_off / 2 + e;  // master element of this bf16 weight
      const float w = master[idx] - step * g;
      master[idx] = w;
      reinterpret_cast<uint16_t*>(packed)[idx] = f32_to_bf16(w);
    } else {
      float* w = reinterpret_cast<float*>(packed + d.packed_off) + e;
      *w = *w - step * g;
    }
  }
}

// master[i] = packed bf16 element i, for i in [off, off + n) (elements).
__global__ __launch_bounds__(256) void master_init_kernel(const uint16_t* __restrict__ packed,
                                                          int64_t off, int64_t n,
                                                          float* __restrict__ master) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) master[off + i] = bf16_to_f32(packed[off + i]);
}

}  // namespace

hipError_t launch_transpose_bf16(const void* in, int64_t ldi, int64_t c0, int rows, int n,
                                 void* out, int64_t ldo, hipStream_t s) {
  if (rows <= 0 || n <= 0) return hipSuccess;
  if (ldo % 8 != 0 || ldo < rows) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((n + kTT - 1) / kTT), (unsigned)((rows + kTT - 1) / kTT));
  hipLaunchKernelGGL(transpose_kernel, grid, dim3(256), 0, s, static_cast<const uint16_t*>(in),
                     ldi, c0, rows, n, static_cast<uint16_t*>(out), ldo);
  return hipGetLastError();
}

hipError_t launch_layernorm_bwd_bf16(const void* x, int64_t ldx, const void* dy, int64_t ldy,
                                     const float* gamma, float eps, int rows, int d, float* dX,
                                     int64_t lddx, void* dXb, int64_t lddxb, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d < 1 || d > 64 * kLnMaxPerLane) return hipErrorInvalidValue;
  hipLaunchKernelGGL(layernorm_bwd_kernel, dim3(grid_for(rows, 4)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(x), ldx, static_cast<const uint16_t*>(dy), ldy,
                     gamma, eps, rows, d, dX, lddx, static_cast<uint16_t*>(dXb), lddxb);
  return hipGetLastError();
}

hipError_t launch_cross_entropy(const float* logits, int64_t ldl, const int32_t* labels, int C,
                                int batch, void* dlogits, int64_t ldd, float* rowloss,
                                hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  hipLaunchKernelGGL(cross_entropy_kernel, dim3((unsigned)batch), dim3(256), 0, s, logits, ldl,
                     labels, C, batch, static_cast<uint16_t*>(dlogits), ldd, rowloss);
  return hipGetLastError();
}

hipError_t launch_rowsum_bf16(const void* in, int64_t ld, int rows, int n, float* out,
                              hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(rowsum_kernel, dim3(grid_for(rows, 4)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(in), ld, rows, n, out);
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float* part, int64_t c_split, int ksplit, int rows, int cols,
                                int64_t ldp, float* out, int64_t ldo, hipStream_t s) {
  const int64_t n = (int64_t)rows * cols;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, part, c_split,
                     ksplit, rows, cols, ldp, out, ldo);
  return hipGetLastError();
}

int growth_sumsq_parts() { return kSqBlocks; }

hipError_t launch_growth_norm(const float* grad, int64_t n, float* part, const float* rowloss,
                              int batch, float clip, float* stats, hipStream_t s) {
  hipLaunchKernelGGL(sumsq_kernel, dim3(kSqBlocks), dim3(256), 0, s, grad, n, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(growth_finish_kernel, dim3(1), dim3(256), 0, s, part, kSqBlocks, rowloss,
                     batch, clip, stats);
  return hipGetLastError();
}

hipError_t launch_growth_update(const GrowthSlice* slices, int nslices, const float* grad,
                                float* master, void* packed, const float* stats, float lr,
                                hipStream_t s) {
  if (nslices <= 0) return hipSuccess;
  hipLaunchKernelGGL(growth_update_kernel, dim3(256, (unsigned)nslices), dim3(256), 0, s, slices,
                     grad, master, static_cast<uint8_t*>(packed), stats, lr);
  return hipGetLastError();
}

hipError_t launch_master_init(const void* packed, int64_t off, int64_t n, float* master,
                              hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(master_init_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(packed), off, n, master);
  return hipGetLastError();
}

}  // namespace elasto
