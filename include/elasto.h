/*
 * elasto.h -- C ABI of the MI355X (gfx950) elastic-ViT inference library.
 *
 * An elastic ViT holds several nested Descendant Networks (DNs) on ONE shared
 * parameter set (Section 4.3; weight sharing, Eq. 8).  A DN mode keeps, per
 * layer, a subset of attention heads and MLP hidden units; because the DNs are
 * nested, every mode's subset is a prefix of one per-layer channel order.
 * The library stores every weight matrix permuted into that order, so a mode
 * reads a contiguous prefix (per row for the K-sliced projections) and never
 * gathers.  A forward in mode k equals a standard ViT forward (Section 4.1:
 * patch embedding, MHA of Eqs. 2-3, GELU MLP of Eq. 5, pre-norm residual
 * blocks, class-token classifier) in which the pruned heads / units are
 * removed, i.e. masked to zero as in Eqs. 4 and 6.  Switching modes
 * (Section 6.2 measures the switch) is a host-side integer store.
 *
 * Conventions for every function:
 *   - All functions are extern "C" and return elasto_status_t (0 = ELASTO_OK)
 *     unless stated otherwise.
 *   - On any error nothing is changed, and elasto_last_error() returns a
 *     message for the calling thread.
 *   - Every argument, config and table check runs before any HIP call, so the
 *     validation paths work without a GPU.
 *   - "device pointer" means memory from hipMalloc (e.g. a torch.cuda tensor's
 *     data_ptr()); "host pointer" means ordinary CPU memory.
 *   - A handle is not thread-safe: use one handle per host thread / stream.
 */
#ifndef ELASTO_H_
#define ELASTO_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct elasto_handle_s* elasto_handle_t;

typedef enum {
  ELASTO_OK = 0,
  ELASTO_ERR_INVALID_ARG = 1,   /* null pointer, bad size, misaligned pointer   */
  ELASTO_ERR_BAD_CONFIG = 2,    /* model shape the library does not support     */
  ELASTO_ERR_BAD_TABLE = 3,     /* DN table inconsistent with the model         */
  ELASTO_ERR_OUT_OF_MEMORY = 4, /* device or host allocation failed             */
  ELASTO_ERR_HIP = 5,           /* a HIP runtime call or kernel launch failed   */
  ELASTO_ERR_MODE_RANGE = 6,    /* mode index outside [0, num_modes)            */
  ELASTO_ERR_BATCH_RANGE = 7,   /* batch outside [1, max_batch]                 */
  ELASTO_ERR_INFEASIBLE = 8     /* no DN meets the selection bounds             */
} elasto_status_t;

/* Arithmetic of the whole path.  BF16: matrices and activations in bf16,
 * MFMA with fp32 accumulation, fp32 LayerNorm / softmax / GELU, fp32 biases
 * and norm parameters; the class-token rows of the residual stream (the only
 * rows the logits depend on at the end) are kept in fp32.  FP32: fp32
 * everywhere (vector-ALU FMA, no reduced-precision matrix mode). */
typedef enum { ELASTO_FP32 = 0, ELASTO_BF16 = 1 } elasto_dtype_t;

/* Model shape.  tokens T = (img/patch)^2 + 1, head_dim = dim/heads.
 * Supported (else ELASTO_ERR_BAD_CONFIG): img % patch == 0, dim % heads == 0,
 * in_chans >= 1, every size >= 1, ln_eps > 0.  BF16 additionally needs
 * head_dim == 64, patch % 8 == 0, dim % 8 == 0 and mlp_hidden % 8 == 0.
 * Both paths need dim <= 2048. */
typedef struct {
  int32_t img, patch, in_chans, dim, depth, heads, mlp_hidden, num_classes;
  int32_t max_batch; /* largest batch a forward may use; scratch is sized for it */
  int32_t dtype;     /* elasto_dtype_t */
  float ln_eps;      /* LayerNorm epsilon (1e-6 for ViT) */
} elasto_config_t;

/* HOST pointers to fp32 weights in canonical PyTorch order ([out, in]);
 * per-layer tensors are stacked on a leading depth axis.  L = depth,
 * d = dim, M = mlp_hidden, C = num_classes, P = patch, T = tokens.
 * qkv_w rows are [q | k | v], each block head-major (head i owns rows
 * i*head_dim .. (i+1)*head_dim-1 of the block); proj_w input columns are
 * head-major the same way.  The caller keeps ownership; the library copies. */
typedef struct {
  const float* patch_w; /* [d][in_chans][P][P] */
  const float* patch_b; /* [d] */
  const float* cls;     /* [d] */
  const float* pos;     /* [T][d] */
  const float* ln1_g;   /* [L][d] */
  const float* ln1_b;   /* [L][d] */
  const float* qkv_w;   /* [L][3d][d] */
  const float* qkv_b;   /* [L][3d] */
  const float* proj_w;  /* [L][d][d] */
  const float* proj_b;  /* [L][d] */
  const float* ln2_g;   /* [L][d] */
  const float* ln2_b;   /* [L][d] */
  const float* fc1_w;   /* [L][M][d] */
  const float* fc1_b;   /* [L][M] */
  const float* fc2_w;   /* [L][d][M] */
  const float* fc2_b;   /* [L][d] */
  const float* norm_g;  /* [d] */
  const float* norm_b;  /* [d] */
  const float* head_w;  /* [C][d] */
  const float* head_b;  /* [C] */
} elasto_weights_t;

/* DN table (HOST pointers, row-major int32).  Mode k, layer l keeps the first
 * n_heads[k][l] heads of head_order[l] and the first n_mlp[k][l] units of
 * mlp_order[l]; prefixes of one order make the modes nested (Eq. 8).
 * Mode 0 conventionally is the widest.  ELASTO_ERR_BAD_TABLE unless:
 * depth == cfg.depth, num_modes >= 1, 1 <= n_heads <= heads,
 * 1 <= n_mlp <= mlp_hidden, and every order row is a permutation.
 *
 * Embedding width (the compress stage also narrows the hidden size of the
 * LayerNorm and patch-embedding layers, Section 4.1): mode k keeps the first
 * n_embed[k] channels of embed_order, the same channels in every layer (the
 * residual stream is shared by all blocks).  Patch embedding, class token and
 * positions produce only those channels, every LayerNorm normalises over
 * them (mean and variance over the n_embed[k] active channels), q/k/v and
 * fc1 read only them, projection and fc2 write only them, and the classifier
 * reads only them; head_dim and the attention scale stay those of the full
 * model.  n_embed == NULL keeps all dim channels in every mode, embed_order ==
 * NULL is the identity.  Needs 1 <= n_embed <= dim (a multiple of 8 on the
 * BF16 path) and embed_order a permutation of dim. */
typedef struct {
  int32_t num_modes, depth;
  const int32_t* n_heads;     /* [num_modes][depth] */
  const int32_t* n_mlp;       /* [num_modes][depth] */
  const int32_t* head_order;  /* [depth][heads] */
  const int32_t* mlp_order;   /* [depth][mlp_hidden] */
  const int32_t* n_embed;     /* [num_modes] or NULL */
  const int32_t* embed_order; /* [dim] or NULL */
} elasto_dn_table_t;

/* ---------------------------------------------------------------- lifecycle */

/* Validates cfg and table, repacks the weights into the prefix layout (bf16
 * rounded to nearest even on the BF16 path), makes one device allocation for
 * the weights and one for max_batch activation scratch, and copies.  The
 * current device at call time owns the handle.  Mode 0 is selected.
 * BF16: also tunes, per DN mode, on the default stream (about a second at
 * ViT-B batch 256; synchronises the device): every GEMM is timed with each
 * tile plan the GEMM kernels offer (at small batches also split-K plans,
 * whose partial products go to the handle's workspace), for forwards of
 * max_batch and of half as many images, and the whole forward is timed
 * against two half-batch forwards of which the second runs on a stream the
 * handle owns (forked from and joined back into the caller's stream with
 * events, so a captured graph captures both).  A forward of more than
 * max_batch / 2 images then runs as chosen.  The choices are kept per
 * process: a later handle of the same configuration, DN widths, max_batch
 * and device takes them without timing.  A handle's outputs are
 * deterministic; handles of different processes may differ within fp32
 * rounding (the plans of the LayerNorm-folded GEMMs round differently).
 * *out receives the handle (unchanged on error). */
elasto_status_t elasto_create(const elasto_config_t* cfg, const elasto_weights_t* w,
                              const elasto_dn_table_t* table, elasto_handle_t* out);

/* Frees all device and host memory of h; waits for nothing (the caller must
 * make sure no enqueued forward still uses h).  h == NULL is accepted. */
elasto_status_t elasto_destroy(elasto_handle_t h);

/* Selects DN mode k for subsequent forwards (Eq. 11 picks k; this applies it).
 * O(1) host store: no HIP call, no weight copy, no synchronisation.  A forward
 * uses the mode current at its enqueue time.  ELASTO_ERR_MODE_RANGE if k is
 * outside [0, num_modes). */
elasto_status_t elasto_set_mode(elasto_handle_t h, int32_t k);
elasto_status_t elasto_get_mode(elasto_handle_t h, int32_t* k);

/* Enqueues one forward in the current mode on hip_stream (a hipStream_t;
 * NULL = default stream) and returns without waiting.
 *   images: device pointer, NCHW [batch][in_chans][img][img], contiguous,
 *           16-byte aligned; bf16 on the BF16 path, fp32 on the FP32 path.
 *   logits: device pointer, fp32 [batch][num_classes].
 * Both stay owned by the caller and must stay valid until the stream work
 * completes.  Allocates nothing and never synchronises; device faults
 * surface at the caller's next synchronisation.  ELASTO_ERR_BATCH_RANGE if
 * batch is outside [1, max_batch]; ELASTO_ERR_HIP if a launch fails. */
elasto_status_t elasto_forward(elasto_handle_t h, const void* images, int32_t batch,
                               float* logits, void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * forward as elasto_forward, with its activation scratch taken from one
 * statically allocated array per GPU instead of the handle's buffers.  The
 * array holds 64 MiB (ELASTO_STATIC_SCRATCH_BYTES), enough for ViT-B/16 at
 * up to 20 images a call; each GPU the library runs on keeps its copy
 * until the process ends.  Allocates nothing (the array's device address is
 * looked up once per device, on the first call there); the caller still
 * passes images and logits as for elasto_forward.
 * Every call on one GPU shares that GPU's array, and a call reads only what
 * it wrote there itself; calls that overlap on one GPU (several streams or
 * several handles at once) race on it and must be serialised by the caller.
 * BATCH_RANGE when batch is outside [1, max_batch] or the batch's
 * activations exceed the array (the message gives both sizes). */
#define ELASTO_STATIC_SCRATCH_BYTES (64LL << 20)
elasto_status_t elasto_forward_static(elasto_handle_t h, const void* images, int32_t batch,
                                      float* logits, void* hip_stream);

/* Thread-local message of the calling thread's last failing call ("" if none).
 * Returns a string, not a status. */
const char* elasto_last_error(void);

/* Work of mode k per image: algorithmic FLOPs (2 x MACs of every contraction,
 * attention included) and bytes of the weight matrices a forward reads. */
elasto_status_t elasto_mode_info(elasto_handle_t h, int32_t k, double* flops_per_image,
                                 int64_t* active_weight_bytes);

/* Device bytes the handle holds: weights (the packed image, plus on the bf16
 * path the LayerNorm-folded copies of the q/k/v and fc1 matrices with their
 * column sums and folded biases per embedding width) and activation scratch. */
elasto_status_t elasto_memory_info(elasto_handle_t h, int64_t* weight_bytes,
                                   int64_t* scratch_bytes);

/* ----------------------------------------------- DN selection (Eq. 11) */
/* Look-up table of the DNs, one entry per mode: each DN is profiled once for
 * its computational cost, latency, memory footprint and accuracy, and the
 * table is consulted at run time (Section 4.4, system monitoring and network
 * selection).  Arrays are host pointers of num_modes doubles; no entry may be
 * NaN.  accuracy and power_w may be NULL (no such data). */
typedef struct {
  int32_t num_modes;
  const double* flops;        /* cost of one forward, any fixed unit           */
  const double* latency_ms;   /* time of one forward                           */
  const double* memory_bytes; /* device memory the DN needs resident           */
  const double* accuracy;     /* user-supplied (no trained weights here)       */
  const double* power_w;      /* power at this cost, from a FLOPs-to-power table */
} elasto_dn_lut_t;

/* Eq. 11: among the modes with latency_ms <= max_latency_ms,
 * memory_bytes <= max_memory_bytes, accuracy >= min_accuracy and, when
 * power_w is given, power_w <= max_power_w, picks the one with the smallest
 * flops; equal flops go to the lower mode index.  Pass +INFINITY (-INFINITY
 * for min_accuracy) to leave a bound open; with accuracy == NULL min_accuracy
 * must be -INFINITY.  *mode = -1 and ELASTO_ERR_INFEASIBLE when no mode meets
 * the bounds; ELASTO_ERR_INVALID_ARG for a NULL table array, num_modes < 1,
 * NaN entries or NaN bounds.  Host only: makes no HIP call. */
elasto_status_t elasto_select_mode(const elasto_dn_lut_t* lut, double max_latency_ms,
                                   double max_memory_bytes, double min_accuracy,
                                   double max_power_w, int32_t* mode);

/* Profiles every mode of the handle at the given batch and fills the cost
 * columns of a selection table (host arrays of num_modes doubles):
 *   latency_ms[k]   median device time of one forward in mode k over `iters`
 *                   forwards after `warmup` untimed ones (HIP events on
 *                   hip_stream; iters in [1, 1000]);
 *   memory_bytes[k] bytes mode k needs resident at this batch: its active
 *                   weight matrices, every fp32 vector parameter, and the
 *                   activation buffers of this batch at the mode's widths;
 *   flops[k]        FLOPs of one forward of `batch` images in mode k.
 * images / logits as for elasto_forward.  Synchronises hip_stream, leaves
 * the handle's mode as it was.  Creates and destroys its own events. */
elasto_status_t elasto_profile_modes(elasto_handle_t h, const void* images, int32_t batch,
                                     float* logits, int32_t warmup, int32_t iters,
                                     void* hip_stream, double* latency_ms,
                                     double* memory_bytes, double* flops);

/* ------------------------------------------------- host-only layout helpers */
/* These make no HIP call; they let a CPU-only caller check validation and the
 * packed prefix layout. */

elasto_status_t elasto_validate(const elasto_config_t* cfg, const elasto_dn_table_t* table);

/* Tensor ids of the packed weight image.  Every axis of length d (embedding
 * channels) is stored in embed_order: packed channel j is canonical channel
 * embed_order[j] (e.g. PATCH_W row j, POS column j, WQKV column j, WO row j). */
typedef enum {
  ELASTO_T_PATCH_W = 0, /* [d][in_chans*P*P], matrix dtype                     */
  ELASTO_T_PATCH_B,     /* [d] fp32                                            */
  ELASTO_T_CLS,         /* [d] fp32                                            */
  ELASTO_T_POS,         /* [T][d] fp32                                         */
  ELASTO_T_NORM_G,      /* [d] fp32                                            */
  ELASTO_T_NORM_B,      /* [d] fp32                                            */
  ELASTO_T_HEAD_W,      /* [C][d], matrix dtype                                */
  ELASTO_T_HEAD_B,      /* [C] fp32                                            */
  ELASTO_T_LN1_G,       /* per layer [d] fp32                                  */
  ELASTO_T_LN1_B,
  ELASTO_T_WQKV,        /* [heads*3*hd][d]: row s*3hd + t*hd + c = qkv_w row
                           t*d + head_order[s]*hd + c (t = q,k,v)              */
  ELASTO_T_BQKV,        /* [heads*3*hd] fp32, same row order                   */
  ELASTO_T_WO,          /* [d][heads*hd]: column s*hd + c = proj_w column
                           head_order[s]*hd + c                                */
  ELASTO_T_BO,          /* [d] fp32                                            */
  ELASTO_T_LN2_G,
  ELASTO_T_LN2_B,
  ELASTO_T_W1,          /* [M][d]: row s = fc1_w row mlp_order[s]              */
  ELASTO_T_B1,          /* [M] fp32, same order                                */
  ELASTO_T_W2,          /* [d][M]: column s = fc2_w column mlp_order[s]        */
  ELASTO_T_B2,          /* [d] fp32                                            */
  ELASTO_T_COUNT
} elasto_tensor_t;

/* Total bytes of the packed weight image for cfg. */
elasto_status_t elasto_packed_bytes(const elasto_config_t* cfg, int64_t* bytes);

/* Byte offset, row count, column count and element size (2 = bf16, 4 = fp32)
 * of one tensor in the packed image; layer is ignored for global tensors. */
elasto_status_t elasto_packed_layout(const elasto_config_t* cfg, int32_t tensor, int32_t layer,
                                     int64_t* offset, int64_t* rows, int64_t* cols,
                                     int32_t* elem_bytes);

/* Writes the packed weight image (exactly what elasto_create copies to the
 * device) into host memory dst of dst_bytes >= elasto_packed_bytes. */
elasto_status_t elasto_pack_weights(const elasto_config_t* cfg, const elasto_weights_t* w,
                                    const elasto_dn_table_t* table, void* dst, int64_t dst_bytes);

/* -------------------------------------------------- per-kernel timing (HIP) */

/* Kernel classes of one forward. */
typedef enum {
  ELASTO_K_PATCH = 0, /* patch-embedding GEMM (+bias, +position, class rows) */
  ELASTO_K_LN,        /* LayerNorm (LN1, LN2, final norm on class rows)      */
  ELASTO_K_QKV,       /* q/k/v GEMM over the active heads                    */
  ELASTO_K_ATTN,      /* fused attention over the active heads               */
  ELASTO_K_PROJ,      /* output projection GEMM + residual add               */
  ELASTO_K_FC1,       /* fc1 GEMM + GELU over the active units               */
  ELASTO_K_FC2,       /* fc2 GEMM + residual add                             */
  ELASTO_K_HEAD,      /* classifier GEMM                                     */
  ELASTO_K_COUNT
} elasto_kernel_t;

/* Starts recording a hipEvent pair around every launch of kernel class kc
 * (kc = -1 stops) for at most max_launches launches; events are created here,
 * not in the forward.  Recording adds two event records per launch. */
elasto_status_t elasto_kernel_timing(elasto_handle_t h, int32_t kc, int32_t max_launches);

/* Waits for the recorded events, returns the summed kernel time (ms) and the
 * launch count since the last read, and resets the accumulation. */
elasto_status_t elasto_kernel_timing_read(elasto_handle_t h, double* total_ms, int64_t* launches);

/* Algorithmic work of one launch of class kc in mode k at the given batch
 * summed over the forward: FLOPs (contractions) and bytes (LayerNorm rows
 * read + written; for contractions the operand and result bytes) and the
 * number of launches of that class in one forward.  On the bf16 path the
 * per-layer LayerNorms are folded into the GEMMs and the LayerNorm class is
 * the final norm of the class-token rows alone. */
elasto_status_t elasto_kernel_work(elasto_handle_t h, int32_t k, int32_t batch, int32_t kc,
                                   double* flops, double* bytes, int32_t* launches);

/* ------------------------------------------- single-kernel entry points */
/* Device-pointer access to the kernels one forward uses, for kernel-level
 * tests.  dtype selects bf16 (MFMA) or fp32 kernels; activations have that
 * dtype, gamma/beta and bias are fp32.  Strides are in elements. */

/* out[r] = LayerNorm(x[r]) * g + b over d features, r < rows.  x row r starts
 * at x + r*x_stride; out is contiguous [rows][d].  BF16 path only: when x_cls
 * is non-NULL, rows with r % tokens == 0 (class-token rows) are read as fp32
 * from x_cls + (r / tokens) * d instead (tokens = 1: every row); d and
 * x_stride must be multiples of 8 and x, out, x_cls, g, b 16-byte aligned.
 * FP32 path: x_cls must be NULL. */
elasto_status_t elasto_op_layernorm(int32_t dtype, const void* x, int64_t x_stride,
                                    const float* x_cls, int32_t tokens, void* out, int64_t rows,
                                    int32_t d, const float* g, const float* b, float eps,
                                    void* hip_stream);

typedef enum {
  ELASTO_EPI_BIAS = 0,     /* C = A W^T + bias                      */
  ELASTO_EPI_BIAS_GELU,    /* C = GELU(A W^T + bias)                */
  ELASTO_EPI_BIAS_RESID,   /* C = C + A W^T + bias (in place)       */
  ELASTO_EPI_BIAS_F32OUT   /* C (fp32) = A W^T + bias               */
} elasto_epilogue_t;

/* C[m][n] = epi(sum_{k<K} A[m*lda + k] * W[n*ldw + k] + bias[n]), m < M,
 * n < N.  Only the first K columns of A / W rows and the first N rows of W
 * are read.  GELU is the erf GELU of Eq. 5 (fp32 path: the device erff;
 * bf16 path: a polynomial form within 1e-4 absolute of it for |z| <= 12 and
 * 1e-4 relative where |GELU(z)| > 0.1, below the bf16 rounding of its
 * result).  BF16 path: lda and ldw multiples of 8, ldc a
 * multiple of 8 (bf16 out) or 4 (fp32 out), A, W, C, bias 16-byte aligned;
 * with ELASTO_EPI_BIAS_RESID a non-NULL C_cls holds the class-token rows
 * (m % tokens == 0) of C in fp32, [M / tokens][N], and those rows of C are
 * neither read nor written.  C_cls must be NULL otherwise. */
elasto_status_t elasto_op_linear(int32_t dtype, int32_t epilogue, const void* A, int64_t lda,
                                 const void* W, int64_t ldw, void* C, int64_t ldc, float* C_cls,
                                 int32_t tokens, const float* bias, int64_t M, int32_t N,
                                 int32_t K, void* hip_stream);

/* The bf16 linear with a LayerNorm folded in, as the forward runs its
 * pre-norm blocks (Section 4.1): the GEMM that writes the residual stream
 * also emits per-row statistics, and the next q/k/v or fc1 GEMM applies the
 * LayerNorm of its input through them instead of a separate pass.
 *
 * Statistics: row m, 64-column segment j (n_j = min(64, width - 64 j)
 * columns) at stats[2 * (m*stats_ld + j)]: the sum of the row's values in the
 * segment, then the sum of their squared deviations from the segment's mean
 * (fp32).  stats_ld is even and >= ceil(width / 64).
 *
 * stats_out != NULL (producer; epilogue ELASTO_EPI_BIAS_RESID): C and C_cls
 * as in elasto_op_linear, and the statistics of every output row over its N
 * columns (width = N, N % 8 == 0), of the values before their rounding to
 * bf16 (class-token rows: of their fp32 values, which are then also written
 * to C, rounded to bf16).
 *
 * stats_in != NULL (consumer; epilogue ELASTO_EPI_BIAS or
 * ELASTO_EPI_BIAS_GELU): with the mean mu_m and biased variance v_m of A's row
 * m over its K columns (width = K), combined from its segments,
 *   C[m][n] = epi(rstd_m * sum_k A[m][k] W[n][k] - rstd_m * mu_m * colsum[n]
 *                 + bias[n]),  rstd_m = 1 / sqrt(v_m + eps),
 * which equals epi(LayerNorm(A[m]) . w_n + b_n) when W holds gamma (.) w,
 * colsum[n] = sum_k W[n][k] and bias[n] = b_n + beta . w_n.
 *
 * Exactly one of stats_out, stats_in is non-NULL; stats are 16-byte
 * aligned; other requirements as for the bf16 elasto_op_linear. */
elasto_status_t elasto_op_linear_ln(int32_t epilogue, const void* A, int64_t lda, const void* W,
                                    int64_t ldw, void* C, int64_t ldc, float* C_cls,
                                    int32_t tokens, const float* bias, int64_t M, int32_t N,
                                    int32_t K, float* stats_out, const float* stats_in,
                                    int64_t stats_ld, const float* colsum, float eps,
                                    void* hip_stream);

/* Multi-head attention (Eq. 3) over `heads` head slots of `batch` sequences
 * of `tokens` rows.  qkv row (b*tokens + t) holds, for slot s, q at columns
 * s*3*hd + [0,hd), k at + [hd,2hd), v at + [2hd,3hd), with row stride
 * qkv_stride; o row holds slot s at columns s*hd + [0,hd), row stride
 * o_stride.  Scores are scaled by `scale`.  BF16 path: head_dim == 64,
 * tokens <= 240, qkv 16-byte aligned with qkv_stride a multiple of 8, o
 * 8-byte aligned with o_stride a multiple of 4 and tokens * o_stride * 2
 * below 2^31. */
elasto_status_t elasto_op_attention(int32_t dtype, const void* qkv, int64_t qkv_stride, void* o,
                                    int64_t o_stride, int32_t batch, int32_t tokens,
                                    int32_t heads, int32_t head_dim, float scale,
                                    void* hip_stream);

/* Convolution of an NHWC bf16 batch, as the elastic ResNet's 3x3 and strided
 * 1x1 layers run it (Section 4.1; a DN mode keeps a prefix of the input
 * channels, i.e. Eq. 7's kernel masks, and reads the first `ca` channels of
 * every tap):
 *   y[(b*Ho + oh)*Wo + ow][j] = relu?(bias[j] + sum over i < kh, jj < kw,
 *       c < ca of x[((b*H + ih)*W + iw)*cs + c] * w[j*ldw + (i*kw + jj)*wseg + c])
 * with ih = oh*stride - pad + i, iw = ow*stride - pad + jj, zero outside the
 * image, Ho = (H + 2*pad - kh)/stride + 1 (Wo likewise), j < n; row stride of
 * y is ldy.  bf16 x, w, y; fp32 bias and accumulation.  cs, ca, wseg, ldw and
 * ldy are multiples of 8, 8 <= ca <= min(cs, wseg), ldw >= kh*kw*wseg, and x,
 * w, y, bias are 16-byte aligned; one image's input and the read part of w
 * must each stay below 2 GiB.  Channels of x at or past ca, and entries of w
 * past ca within each tap segment, are never used. */
elasto_status_t elasto_op_conv2d(const void* x, int32_t batch, int32_t H, int32_t W, int32_t cs,
                                 int32_t ca, int32_t kh, int32_t kw, int32_t stride, int32_t pad,
                                 const void* w, int64_t ldw, int64_t wseg, const float* bias,
                                 void* y, int64_t ldy, int32_t n, int32_t relu, void* hip_stream);

/* ================================================ growth step (Section 4.2) */
/* Growing DN mode k re-introduces the weights mode k holds and the next
 * smaller mode k + 1 (the previous level) lacks; mode k + 1's weights are
 * shared and frozen.  With the prefix layout the re-introduced weights of
 * layer l are contiguous slices: q/k/v rows and biases of head slots
 * [n_heads[k+1][l], n_heads[k][l]), the output projection's columns of
 * those slots, fc1 rows and biases and fc2 columns of MLP units
 * [n_mlp[k+1][l], n_mlp[k][l]).  Eq. 9's gradient mask G is 1 exactly there. */
typedef struct elasto_growth_s* elasto_growth_t;

/* Growth context of a bf16 handle for batches of up to max_batch images:
 * fp32 master copies of the trainable matrices (initialised from the
 * handle's bf16 weights), the activations one step keeps and the gradient
 * buffers, all in device memory allocated here (on the handle's device).
 * The handle must outlive the context.  BAD_CONFIG: not a bf16 handle, or
 * head_dim != 64. */
elasto_status_t elasto_growth_create(elasto_handle_t h, int32_t max_batch, elasto_growth_t* out);
elasto_status_t elasto_growth_destroy(elasto_growth_t g);

/* One growth step of mode k (Section 4.2: Eq. 9 and the selective gradient
 * clipping): the mode-k forward of `batch` images (device, as for
 * elasto_forward), the mean cross-entropy against labels (device int32
 * [batch], each in [0, num_classes); another value makes the loss NaN), the
 * backward, G (.) grad for the re-introduced slices only, scaled by
 * min(1, clip_norm / |G (.) grad|_2), and W <- W - lr * that, applied to
 * the fp32 masters and stored, rounded to bf16 (biases: fp32), into the
 * handle's packed weights.  Every weight of mode k + 1 stays bit-identical.
 * Needs 0 <= k < num_modes - 1, n_heads / n_mlp of mode k + 1 at most those
 * of mode k in every layer, and the full embedding width in modes k and
 * k + 1; lr finite, clip_norm > 0 (INFINITY: no clipping).  stats: device
 * float[3] (or NULL) receiving mean loss, |G (.) grad|_2 and the clip
 * factor.  Enqueued on hip_stream without synchronising; the handle's
 * forward must not run on another stream meanwhile. */
elasto_status_t elasto_growth_step(elasto_growth_t g, int32_t mode, const void* images,
                                   const int32_t* labels, int32_t batch, float lr,
                                   float clip_norm, float* stats, void* hip_stream);

/* Synchronous copy to host memory: which = 0 the handle's packed weights
 * (elasto_packed_bytes long), which = 1 the fp32 masters (one float per
 * bf16 element of the packed image: float i mirrors the bf16 element at
 * byte 2i; only the re-trainable matrices, WQKV, WO, W1 and W2, are kept).
 * bytes must equal the full size. */
elasto_status_t elasto_growth_read(elasto_growth_t g, int32_t which, void* host_dst,
                                   int64_t bytes);

/* ======================================== elastic bottleneck ResNet (CNN) */
/* The paper applies the same elastic transformation to CNNs (Eq. 7 masks
 * whole convolution kernels; Table 2 reports ResNet-50 DNs).  This is the
 * inference forward of a ResNet-50-style network (7x7 stride-2 stem + ReLU,
 * 3x3 stride-2 max pool, bottleneck blocks of 1x1 reduce, 3x3 with the block
 * stride and 1x1 expand, a 1x1 projection shortcut with the same stride on
 * each stage's first block, ReLU after the sum, global average pooling,
 * linear classifier), BF16 only: bf16 NHWC activations, MFMA convolutions
 * (implicit GEMMs: each tile's input patches are loaded straight from the
 * activation, no patch matrix is written), fp32 biases and logits.  Batch
 * norm at inference is a per-channel affine map: the caller folds it into
 * each convolution's weights and bias.
 *
 * A DN mode keeps, in each bottleneck, the first n_width[k][b] filters of
 * the 1x1 reduce (in order1) and of the 3x3 (in order2); a pruned filter
 * also removes the input channels that read it.  The weights are stored in
 * those orders so a mode reads prefixes (nested DNs, Eq. 8). */
typedef struct elasto_cnn_s* elasto_cnn_t;

/* Shape.  Blocks: blocks[s] bottlenecks in stage s, inner width widths[s],
 * output channels widths[s] * expansion; stage s > 0 starts with stride 2.
 * Needs img % 32 == 0, stem, widths[] and expansion * widths[] multiples of
 * 8, 1 <= num_stages <= 8, 1 <= in_chans <= 4 (image channels), dtype ==
 * ELASTO_BF16. */
typedef struct {
  int32_t img, in_chans, stem, num_stages;
  int32_t widths[8], blocks[8];
  int32_t expansion, num_classes, max_batch, dtype;
} elasto_cnn_config_t;

/* HOST pointers to fp32 tensors in PyTorch order, in this sequence:
 * stem_w [stem][in_chans][7][7], stem_b; then per block b (stage-major):
 * c1_w [w][c_in][1][1], c1_b, c2_w [w][w][3][3], c2_b, c3_w [c_out][w][1][1],
 * c3_b, and on each stage's first block dn_w [c_out][c_in][1][1], dn_b;
 * then fc_w [classes][features], fc_b.  num_tensors must match. */
typedef struct {
  int32_t num_tensors;
  const float* const* tensors;
} elasto_cnn_weights_t;

/* n_width [num_modes][num_blocks], each a multiple of 8 in [8, width];
 * order1 / order2: the blocks' filter orders concatenated (block b holds a
 * permutation of its width).  ELASTO_ERR_BAD_TABLE otherwise. */
typedef struct {
  int32_t num_modes, num_blocks;
  const int32_t* n_width;
  const int32_t* order1;
  const int32_t* order2;
} elasto_cnn_table_t;

/* Host-only validation (no HIP call). */
elasto_status_t elasto_cnn_validate(const elasto_cnn_config_t* cfg, const elasto_cnn_table_t* t);

/* As elasto_create: validates, packs (bf16; a 3x3 filter row holds its 9
 * taps one after another, each tap's input channels in order1 order over the
 * block's full width, so a narrower mode's channels are a prefix of every
 * tap's segment), one weight and one scratch allocation sized for max_batch,
 * mode 0 selected.  With max_batch >= 32 it also tunes as elasto_create
 * does: tile plans of each convolution of every DN mode, for whole and
 * half-batch forwards, and whether a mode runs as two half-batch forwards on
 * two streams (about two seconds for ResNet-50 at 256 images; synchronises
 * the device), kept per process for handles of the same shapes; forwards of
 * more than max_batch / 2 images run as chosen.  Every choice gives
 * bit-identical outputs. */
elasto_status_t elasto_cnn_create(const elasto_cnn_config_t* cfg, const elasto_cnn_weights_t* w,
                                  const elasto_cnn_table_t* table, elasto_cnn_t* out);
elasto_status_t elasto_cnn_destroy(elasto_cnn_t h);
elasto_status_t elasto_cnn_set_mode(elasto_cnn_t h, int32_t k);  /* O(1) host store */
elasto_status_t elasto_cnn_get_mode(elasto_cnn_t h, int32_t* k);

/* One forward in the current mode on hip_stream: images bf16 NCHW
 * [batch][in_chans][img][img] (device, 16-byte aligned), logits fp32
 * [batch][num_classes] (device).  Allocates nothing, never synchronises. */
elasto_status_t elasto_cnn_forward(elasto_cnn_t h, const void* images, int32_t batch,
                                   float* logits, void* hip_stream);

/* Multiply-accumulates per image of mode k (convolutions and classifier) and
 * bytes of the filters and classifier the mode reads. */
elasto_status_t elasto_cnn_mode_info(elasto_cnn_t h, int32_t k, double* macs_per_image,
                                     int64_t* active_weight_bytes);

#ifdef __cplusplus
}
#endif

#endif /* ELASTO_H_ */
