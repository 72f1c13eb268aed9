// Internal launchers of the gfx950 kernels (host-side declarations).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace elasto {

// Output element types: Bias, BiasGelu, BiasResid and Patch write the path's
// activation type; BiasF32 writes fp32.  On the bf16 path the residual stream
// (BiasResid, Patch) keeps its class-token rows (row % tokens == 0) in fp32
// in `ccls` ([rows / tokens][N]) when that pointer is given.
enum class Epi : int {
  Bias = 0,      // C = acc + bias
  BiasGelu = 1,  // C = GELU(acc + bias)
  BiasResid = 2, // C = C + acc + bias (in place)
  BiasF32 = 3,   // C (fp32) = acc + bias
  Patch = 4,     // patch embedding: A rows are image patches (row t == 0 of
                 // each sequence is the class row), C = acc + (cls|bias) + pos
  GeluBwd = 5,   // C = acc * GELU'(aux) (aux: the pre-activation, bf16)
};

// C[m][n] = epi(sum_k A[m][k] W[n][k] + bias[n]).
struct GemmArgs {
  const void* A = nullptr;
  int64_t lda = 0;
  const void* W = nullptr;
  int64_t ldw = 0;
  void* C = nullptr;
  int64_t ldc = 0;
  const float* bias = nullptr;
  int64_t M = 0;
  int N = 0;
  int K = 0;
  // Patch loader: A row m = b*tokens + t reads patch t-1 of image b.
  const void* img = nullptr;
  int img_size = 0, patch = 0, chans = 0, grid = 0, tokens = 0;
  const float* cls = nullptr;
  const float* pos = nullptr;
  int64_t ldpos = 0;  // row stride of pos (elements); 0: N
  float* ccls = nullptr;
  bool relu = false;  // bf16 Bias / BiasResid epilogues: max(result, 0)
  // BiasResid: residual read from res (row stride ldres) instead of C.
  const void* res = nullptr;
  int64_t ldres = 0;
  // BiasGelu: also store the pre-activation to aux (bf16); GeluBwd: read it.
  void* aux = nullptr;
  int64_t ldaux = 0;
  // BiasF32 only: split K into ksplit chunks of kchunk (a multiple of 64);
  // chunk i writes its partial product to C + i * c_split (fp32 elements).
  int ksplit = 1, kchunk = 0;
  int64_t c_split = 0;
  // LayerNorm folded into the GEMMs (bf16 path).
  // Producer (BiasResid, Patch): ln_out != nullptr also writes, for every
  // output row r and every 64-column segment j of [0, N), the pair (sum of
  // the row's values there, sum of their squared deviations from the
  // segment's mean), of the values before their rounding to bf16, to
  // ln_out[r * ln_ld + j] (ln_ld even, >= ceil(N / 64); class-token rows:
  // of their fp32 values, which are then also stored rounded to bf16 in C).
  // Needs N % 8 == 0.
  // Consumer (Bias, BiasGelu): ln_in != nullptr treats A as the LayerNorm
  // input: with mean mu_r and rstd r_r of A's row r over its K columns
  // (the ceil(K / 64) segments of ln_in, same layout, merged pairwise; the
  // last segment has K - 64 * (ceil(K / 64) - 1) columns) the result is
  // epi(r_r * (A W^T)[r][n] - r_r * mu_r * ln_colsum[n] + bias[n]), i.e.
  // LN(A) W^T + bias when W holds gamma (x) the weights, ln_colsum[n] the sum
  // of W's row n over its K columns and bias the original bias plus
  // beta . W.
  float2* ln_out = nullptr;
  const float2* ln_in = nullptr;
  int64_t ln_ld = 0;
  const float* ln_colsum = nullptr;
  float ln_eps = 0.0f;
  // Bias, BiasGelu, BiasResid (bf16, no relu / aux): a device workspace of
  // ws_bytes (256-byte aligned) lets a launch whose 128x128 tiles would fill
  // under half the CUs split K into chunks whose fp32 partial products go
  // there, summed by a second kernel that applies the epilogue.  At most
  // kSplitWsBytes is ever used.
  float* ws = nullptr;
  int64_t ws_bytes = 0;
  // Tile plan (see kTilePlans): 0 lets the planner choose; another value
  // runs that one configuration, or returns hipErrorNotSupported where it
  // cannot take these arguments.
  int plan = 0;
};

// Tile plans a caller may force (GemmArgs::plan, ConvArgs::plan): 1 256x256,
// 2 256x128, 3 128x128, 4 256x64, 5 128x128 with four LDS stages (bf16
// Bias / BiasGelu / BiasResid, no implicit convolution, K a multiple of 64
// and >= 256), 6 the persistent 256x256 kernel (where the planner may use
// it).  Every plan walks K in the same order with the same MFMA
// instruction, so for a GEMM with no LayerNorm work (ln_in, ln_out) and no
// class-token rows (ccls) the outputs are bit-identical whatever the plan.
// Plans kSplitPlan0 + i split K into about kSplitChunks[i] chunks (bf16 Bias /
// BiasGelu / BiasResid with a workspace, where the 128x128 tiles would fill
// under half the CUs; the partials are summed in chunk order, so the bits
// differ from the unsplit plans').  A forced tile plan (1-6) never splits;
// plan 0 splits where the planner's cost model says so.
constexpr int kSplitPlan0 = 7;
constexpr int kSplitChunks[] = {2, 3, 4, 6, 8, 12, 16};
constexpr int kTilePlans = kSplitPlan0 + (int)(sizeof(kSplitChunks) / sizeof(kSplitChunks[0]));

// Largest split-K workspace the planner uses: chunks are limited to the CU
// count over the 128x128 tile count, so chunks x M x N stays below
// 256 x 128 x 128 fp32 values.
constexpr int64_t kSplitWsBytes = (int64_t)256 * 128 * 128 * 4;

hipError_t launch_gemm_bf16(Epi epi, const GemmArgs& a, hipStream_t s);

// Implicit-GEMM convolution, bf16, Bias epilogue (optional ReLU):
// C[(n, oh, ow)][j] = sum_{tap, c < Ca} x[n][ih][iw][c] * weight[j][tap*wseg + c] + bias[j]
// with (ih, iw) = (oh*stride - pad + tap/KW, ow*stride - pad + tap%KW), zero
// outside the image.  x NHWC with channel stride Cs; C rows of ldc elements.
// row_window > 0 (KW = 1, pad = 0): tap i reads the Ca elements from pixel
// (oh*stride + i, ow*stride) on, a window of Ca / Cs pixels along the row
// (the caller keeps it inside the row); the output width is then
// (W - row_window) / stride + 1.
struct ConvArgs {
  const void* x = nullptr;
  int batch = 0, H = 0, W = 0, Cs = 0, Ca = 0;
  int KH = 1, KW = 1, stride = 1, pad = 0;
  const void* weight = nullptr;
  int64_t ldw = 0, wseg = 0;
  void* C = nullptr;
  int64_t ldc = 0;
  const float* bias = nullptr;
  int N = 0;
  bool relu = false;
  int row_window = 0;
  int plan = 0;  // as GemmArgs::plan (the persistent and four-stage plans do not apply)
};
hipError_t launch_conv_bf16(const ConvArgs& a, hipStream_t s);
hipError_t launch_gemm_f32(Epi epi, const GemmArgs& a, hipStream_t s);

// out[r] = LN(x[r]) over d features; x row stride x_stride, out contiguous.
// bf16 variant: x is bf16, except that rows with r % tokens == 0 read fp32
// xcls + (r / tokens) * d when xcls is given (the class-token rows).
hipError_t launch_layernorm_bf16(const void* x, int64_t x_stride, const float* xcls, int tokens,
                                 void* out, int64_t rows, int d, const float* g, const float* b,
                                 float eps, hipStream_t s);
hipError_t launch_layernorm_f32(const void* x, int64_t x_stride, void* out, int64_t rows, int d,
                                const float* g, const float* b, float eps, hipStream_t s);

struct AttnArgs {
  const void* qkv = nullptr;
  int64_t qkv_stride = 0;
  void* o = nullptr;
  int64_t o_stride = 0;
  int batch = 0, tokens = 0, heads = 0, head_dim = 0;
  float scale = 1.0f;
};

hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t s);
hipError_t launch_attention_f32(const AttnArgs& a, hipStream_t s);

// Backward of launch_attention_bf16 (head_dim 64): from qkv (the forward's
// input) and dout (gradient of o, slot s at columns s*64, row stride
// dout_stride) write dq, dk, dv into dqkv, laid out like qkv.  stats holds
// batch*heads*tokens*2 floats of scratch (per-query softmax statistics).
struct AttnBwdArgs {
  const void* qkv = nullptr;
  int64_t qkv_stride = 0;
  const void* dout = nullptr;
  int64_t dout_stride = 0;
  void* dqkv = nullptr;
  int64_t dqkv_stride = 0;
  float* stats = nullptr;
  int batch = 0, tokens = 0, heads = 0, head_dim = 0;
  float scale = 1.0f;
};
hipError_t launch_attention_bwd_bf16(const AttnBwdArgs& a, hipStream_t s);

// Growth-step helpers (growth_kernels.hip).
// out[c][r] = in[r][c0 + c], r < rows, c < n (bf16; ldo % 8 == 0, ldo >= rows).
hipError_t launch_transpose_bf16(const void* in, int64_t ldi, int64_t c0, int rows, int n,
                                 void* out, int64_t ldo, hipStream_t s);
// LayerNorm backward (gamma only; beta and gamma are not trained): from x
// (the LN input, bf16) and dy (bf16), dX[r] += dx (fp32) and dXb[r] = bf16(dX[r]).
hipError_t launch_layernorm_bwd_bf16(const void* x, int64_t ldx, const void* dy, int64_t ldy,
                                     const float* gamma, float eps, int rows, int d, float* dX,
                                     int64_t lddx, void* dXb, int64_t lddxb, hipStream_t s);
// Mean cross-entropy pieces: dlogits (bf16) = (softmax - onehot) / batch and
// the per-image loss (NaN for a label outside [0, C)).
hipError_t launch_cross_entropy(const float* logits, int64_t ldl, const int32_t* labels, int C,
                                int batch, void* dlogits, int64_t ldd, float* rowloss,
                                hipStream_t s);
hipError_t launch_rowsum_bf16(const void* in, int64_t ld, int rows, int n, float* out,
                              hipStream_t s);
hipError_t launch_splitk_reduce(const float* part, int64_t c_split, int ksplit, int rows, int cols,
                                int64_t ldp, float* out, int64_t ldo, hipStream_t s);
// stats[0..2] = mean loss, L2 norm of grad[0, n), clip factor min(1, clip / norm);
// part holds growth_sumsq_parts() floats of scratch.
int growth_sumsq_parts();
hipError_t launch_growth_norm(const float* grad, int64_t n, float* part, const float* rowloss,
                              int batch, float clip, float* stats, hipStream_t s);
// One trainable slice of the packed weights: rows x cols elements from byte
// packed_off with row stride ld (elements); its gradient at grad + grad_off
// with row stride grad_ld.  bf16 slices update the fp32 master element of
// the same index (packed byte offset / 2) and store its rounding.
struct GrowthSlice {
  int64_t packed_off, ld, grad_off;
  int32_t grad_ld, rows, cols, is_bf16;
};
hipError_t launch_growth_update(const GrowthSlice* slices, int nslices, const float* grad,
                                float* master, void* packed, const float* stats, float lr,
                                hipStream_t s);
hipError_t launch_master_init(const void* packed, int64_t off, int64_t n, float* master,
                              hipStream_t s);

// Weights of a LayerNorm folded into the following linear layer (bf16):
// for n < N, Wf[n][k] = bf16(gamma[k] * W[n][k]) for k < D, and for every
// width e = widths[w] (w < nw), colsum[w * ldv + n] = sum_{k<e} Wf[n][k] and
// cbias[w * ldv + n] = bias[n] + sum_{k<e} beta[k] * W[n][k].  W and Wf have
// row stride D (bf16).
hipError_t launch_ln_fold(const void* W, int N, int D, const float* gamma, const float* beta,
                          const float* bias, const int32_t* widths, int nw, void* Wf,
                          float* colsum, float* cbias, int64_t ldv, hipStream_t s);

// Largest token count the bf16 attention kernel supports (K and V of one
// head are staged whole in LDS).
constexpr int kAttnMaxTokens = 240;

// Elastic bottleneck-ResNet data movement (conv.hip).  NHWC bf16.
hipError_t launch_pad_nhwc4(const void* img, int batch, int C, int H, int W, int pad, void* out,
                            hipStream_t s);
// Stem + max pool of the bottleneck ResNet in one launch: NCHW bf16 images
// (C <= 4 channels, S x S, S % 32 == 0), packed stem filters [N][ldw] bf16
// (kernel row i, column j < 8, channel c < 4 at i*32 + j*4 + c; column 7
// and channels >= C zero), fp32 bias, out NHWC [batch][S/4][S/4][N] bf16.
// N is 32 or 64.
hipError_t launch_stem_pool(const void* img, int batch, int C, int S, const void* w, int ldw,
                            const float* bias, int N, void* out, hipStream_t s);
hipError_t launch_max_pool_3x3_s2(const void* x, int batch, int H, int W, int C, void* y,
                                  hipStream_t s);
hipError_t launch_avg_pool(const void* x, int batch, int HW, int C, void* y, hipStream_t s);

// Statically allocated activation scratch (static_scratch.hip): its size, and
// the device address of the current device's copy (looked up on the first
// call per device; later calls return the cached address).
constexpr int64_t kStaticScratchBytes = (int64_t)64 << 20;
hipError_t static_scratch(void** ptr, int64_t* bytes);

}  // namespace elasto
