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
};

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

// Largest token count the bf16 attention kernel supports (K and V^T of one
// head are staged whole in LDS).
constexpr int kAttnMaxTokens = 240;

// Elastic bottleneck-ResNet data movement (conv.hip).  NHWC bf16.
hipError_t launch_pad_nhwc4(const void* img, int batch, int C, int H, int W, int pad, void* out,
                            hipStream_t s);
hipError_t launch_max_pool_3x3_s2(const void* x, int batch, int H, int W, int C, void* y,
                                  hipStream_t s);
hipError_t launch_avg_pool(const void* x, int batch, int HW, int C, void* y, hipStream_t s);

}  // namespace elasto
