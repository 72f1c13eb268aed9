// C ABI of the growth step (Section 4.2, Eq. 9 and the selective gradient
// clipping) on a bf16 ViT handle.
//
// One step of mode k (h_l = n_heads[k][l], m_l = n_mlp[k][l]; hp_l, mp_l
// those of mode k + 1; M = batch * tokens rows):
//   forward of mode k keeping, per layer, the block input X_l, LN outputs
//   u1 / u2, qkv, the attention output o, the mid-block stream Xm_l, and the
//   fc1 pre-activation and GELU output; the residual stream is bf16 in all
//   rows (class rows included);
//   cross-entropy -> dlogits; head backward -> d(class LN output);
//   final LN backward into the fp32 stream gradient dX (class rows);
//   per layer, last to first:
//     fc2:  dh = (dX W2[:, :m]) * GELU'(pre)     (GEMM, GELU' epilogue)
//           dW2[:, mp:m] = dX^T g[:, mp:m]        (transposes + split-K GEMM)
//     fc1:  du = dh W1[:m]; dW1[mp:m] = dh[:, mp:m]^T u2; db1 = column sums
//     LN2 backward: dX += LN'(du)
//     proj: do = dX WO[:, :64h]; dWO[:, 64hp:64h] = dX^T o[:, 64hp:64h]
//     attention backward -> dqkv
//     qkv:  du = dqkv WQKV[:192h]; dWQKV[192hp:192h] = dqkv[:, ...]^T u1; dbqkv
//     LN1 backward: dX += LN'(du)
//   |G (.) grad| over the gradients of the re-introduced slices (which is all
//   G keeps), clip factor, masked update of fp32 masters -> packed bf16.
// Weight gradients of shared (frozen) weights are never formed: with the
// prefix layout, G selects contiguous slices, so the gradient GEMMs run over
// those slices only.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "handle.h"
#include "kernels.h"
#include "layout.h"

using namespace elasto;

namespace {

int64_t al256(int64_t v) { return (v + 255) / 256 * 256; }
int64_t up8(int64_t v) { return (v + 7) / 8 * 8; }
int64_t up4(int64_t v) { return (v + 3) / 4 * 4; }

// Gradient offsets (floats) of one layer's slices in the gradient arena.
struct LayerPlan {
  int h, hp, m, mp;
  int64_t qkvw, qkvb, proj, fc1w, fc1b, fc2w;
};

struct ModePlan {
  std::vector<LayerPlan> layers;
  int64_t grad_floats = 0;
  GrowthSlice* slices = nullptr;  // device
  int nslices = 0;
};

}  // namespace

struct elasto_growth_s {
  elasto_handle_s* h = nullptr;
  int device = 0;
  int max_batch = 0;
  int64_t Mmax = 0, Mp8 = 0;
  uint8_t* mem = nullptr;
  int64_t mem_bytes = 0;
  float* master = nullptr;
  std::vector<uint16_t*> X, Xm, u1, u2, qkv, o, pre, gact;
  uint16_t *ucls = nullptr, *dlog = nullptr, *ducls = nullptr, *dXb = nullptr, *du = nullptr,
           *dh = nullptr, *dout = nullptr, *dqkv = nullptr, *TA = nullptr, *TB = nullptr,
           *WT = nullptr, *WhT = nullptr;
  float *logits = nullptr, *rowloss = nullptr, *dX = nullptr, *part = nullptr, *grad = nullptr,
        *sq = nullptr, *stats = nullptr, *astats = nullptr;
  int64_t part_floats = 0;
  int ldlog = 0, ldlogits = 0;
  std::vector<ModePlan> plans;  // per k < num_modes - 1 (empty layers when not growable)
};

namespace {

const uint8_t* Wb(const elasto_handle_s* h, int id, int layer = 0) {
  return h->dw + h->lay.get(id, layer).offset;
}
const float* Fp(const elasto_handle_s* h, int id, int layer = 0) {
  return reinterpret_cast<const float*>(Wb(h, id, layer));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Modes k and k + 1 can be grown from one to the other.
bool growable(const elasto_handle_s* h, int k, const char** why) {
  const int L = h->cfg.depth;
  if (h->n_embed[k] != h->cfg.dim || h->n_embed[k + 1] != h->cfg.dim) {
    *why = "growth needs the full embedding width in modes k and k + 1";
    return false;
  }
  for (int l = 0; l < L; ++l)
    if (h->n_heads[(size_t)(k + 1) * L + l] > h->n_heads[(size_t)k * L + l] ||
        h->n_mlp[(size_t)(k + 1) * L + l] > h->n_mlp[(size_t)k * L + l]) {
      *why = "mode k + 1 is not nested in mode k";
      return false;
    }
  return true;
}

}  // namespace

extern "C" {

elasto_status_t elasto_growth_create(elasto_handle_t h, int32_t max_batch, elasto_growth_t* out) {
  if (!h || !out) return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  *out = nullptr;
  const elasto_config_t& c = h->cfg;
  if (c.dtype != ELASTO_BF16) return fail(ELASTO_ERR_BAD_CONFIG, "growth steps need a bf16 handle");
  if (h->dims.hd != 64) return fail(ELASTO_ERR_BAD_CONFIG, "growth steps need head_dim 64");
  if (max_batch < 1 || (int64_t)max_batch * h->dims.T >= ((int64_t)1 << 30))
    return fail(ELASTO_ERR_INVALID_ARG, "max_batch %d out of range", max_batch);
  elasto_growth_s* g = new (std::nothrow) elasto_growth_s();
  if (!g) return fail(ELASTO_ERR_OUT_OF_MEMORY, "host allocation failed");
  g->h = h;
  g->device = h->device;
  g->max_batch = max_batch;
  const int L = c.depth, D = c.dim, Mh = c.mlp_hidden, C = c.num_classes, T = h->dims.T;
  g->Mmax = (int64_t)max_batch * T;
  g->Mp8 = up8(g->Mmax);
  const int64_t M = g->Mmax, B = max_batch;
  g->ldlog = (int)up8(C);
  g->ldlogits = (int)up4(C);

  // Per-mode plans: gradient arena offsets and update slices.
  std::vector<std::vector<GrowthSlice>> host_slices;
  int64_t grad_max = 0, slice_max = 0;
  g->plans.resize(h->num_modes > 1 ? h->num_modes - 1 : 0);
  for (int k = 0; k + 1 < h->num_modes; ++k) {
    ModePlan& mp = g->plans[k];
    std::vector<GrowthSlice> sl;
    const char* why = nullptr;
    if (growable(h, k, &why)) {
      int64_t off = 0;
      for (int l = 0; l < L; ++l) {
        LayerPlan lp;
        lp.h = h->n_heads[(size_t)k * L + l];
        lp.hp = h->n_heads[(size_t)(k + 1) * L + l];
        lp.m = h->n_mlp[(size_t)k * L + l];
        lp.mp = h->n_mlp[(size_t)(k + 1) * L + l];
        const int64_t dq = 192LL * (lp.h - lp.hp), dm = lp.m - lp.mp;
        lp.qkvw = off; off += dq * D;
        lp.qkvb = off; off += dq;
        lp.proj = off; off += (int64_t)D * 64 * (lp.h - lp.hp);
        lp.fc1w = off; off += dm * D;
        lp.fc1b = off; off += dm;
        lp.fc2w = off; off += (int64_t)D * dm;
        mp.layers.push_back(lp);
        slice_max = std::max(slice_max, std::max(dq * D, dm * D));
        auto add = [&](int id, int64_t origin_bytes, int64_t ld, int rows, int cols, int64_t goff,
                       int gld, int bf) {
          if (rows <= 0 || cols <= 0) return;
          GrowthSlice s;
          s.packed_off = h->lay.get(id, l).offset + origin_bytes;
          s.ld = ld; s.rows = rows; s.cols = cols; s.grad_off = goff; s.grad_ld = gld; s.is_bf16 = bf;
          sl.push_back(s);
        };
        add(ELASTO_T_WQKV, 192LL * lp.hp * D * 2, D, (int)dq, D, lp.qkvw, D, 1);
        add(ELASTO_T_BQKV, 192LL * lp.hp * 4, 0, 1, (int)dq, lp.qkvb, 0, 0);
        add(ELASTO_T_WO, 64LL * lp.hp * 2, D, D, 64 * (lp.h - lp.hp), lp.proj, 64 * (lp.h - lp.hp), 1);
        add(ELASTO_T_W1, (int64_t)lp.mp * D * 2, D, (int)dm, D, lp.fc1w, D, 1);
        add(ELASTO_T_B1, (int64_t)lp.mp * 4, 0, 1, (int)dm, lp.fc1b, 0, 0);
        add(ELASTO_T_W2, (int64_t)lp.mp * 2, Mh, D, (int)dm, lp.fc2w, (int)dm, 1);
      }
      mp.grad_floats = off;
      grad_max = std::max(grad_max, off);
    }
    mp.nslices = (int)sl.size();
    host_slices.push_back(std::move(sl));
  }
  // Split-K partials: up to kMaxSplit chunks of the largest slice.
  const int kMaxSplit = 32;
  g->part_floats = kMaxSplit * std::max<int64_t>(up4(std::max(3 * D, Mh)) * D, 1);
  (void)slice_max;

  // One device block for everything.
  const int64_t MD = M * D * 2;
  std::vector<int64_t> sizes;
  auto want = [&](int64_t bytes) { sizes.push_back(al256(std::max<int64_t>(bytes, 1))); return sizes.size() - 1; };
  const size_t i_master = want(h->lay.total / 2 * 4);
  const size_t i_X = want(MD * (L + 1)), i_Xm = want(MD * L), i_u1 = want(MD * L), i_u2 = want(MD * L),
               i_qkv = want(M * 3 * D * 2 * L), i_o = want(MD * L), i_pre = want(M * Mh * 2 * L),
               i_g = want(M * Mh * 2 * L);
  const size_t i_ucls = want(B * D * 2), i_logits = want(B * g->ldlogits * 4),
               i_dlog = want(B * g->ldlog * 2), i_ducls = want(B * D * 2), i_rowloss = want(B * 4),
               i_dX = want(M * D * 4), i_dXb = want(MD), i_du = want(MD), i_dh = want(M * Mh * 2),
               i_dout = want(MD), i_dqkv = want(M * 3 * D * 2), i_TA = want(D * g->Mp8 * 2),
               i_TB = want((int64_t)std::max(Mh, 3 * D) * g->Mp8 * 2),
               i_WT = want((int64_t)std::max(3 * D, Mh) * D * 2), i_WhT = want((int64_t)D * g->ldlog * 2),
               i_part = want(g->part_floats * 4), i_grad = want(grad_max * 4),
               i_sq = want((int64_t)growth_sumsq_parts() * 4), i_stats = want(4 * 4),
               i_astats = want((int64_t)B * h->cfg.heads * T * 2 * 4);
  int64_t slice_bytes = 0;
  for (const auto& v : host_slices) slice_bytes += al256((int64_t)v.size() * sizeof(GrowthSlice));
  const size_t i_slices = want(slice_bytes);
  int64_t total = 0;
  std::vector<int64_t> offs(sizes.size());
  for (size_t i = 0; i < sizes.size(); ++i) { offs[i] = total; total += sizes[i]; }

  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
    if (hipSetDevice(h->device) != hipSuccess) { delete g; return fail(ELASTO_ERR_HIP, "cannot select device"); }
  }
  if (hipMalloc(reinterpret_cast<void**>(&g->mem), (size_t)total) != hipSuccess) {
    (void)hipGetLastError();
    delete g;
    return fail(ELASTO_ERR_OUT_OF_MEMORY, "device allocation of %lld bytes failed", (long long)total);
  }
  g->mem_bytes = total;
  auto at = [&](size_t i) { return g->mem + offs[i]; };
  auto bf = [&](size_t i) { return reinterpret_cast<uint16_t*>(at(i)); };
  auto fl = [&](size_t i) { return reinterpret_cast<float*>(at(i)); };
  g->master = fl(i_master);
  for (int l = 0; l <= L; ++l) g->X.push_back(bf(i_X) + (int64_t)l * M * D);
  for (int l = 0; l < L; ++l) {
    g->Xm.push_back(bf(i_Xm) + (int64_t)l * M * D);
    g->u1.push_back(bf(i_u1) + (int64_t)l * M * D);
    g->u2.push_back(bf(i_u2) + (int64_t)l * M * D);
    g->qkv.push_back(bf(i_qkv) + (int64_t)l * M * 3 * D);
    g->o.push_back(bf(i_o) + (int64_t)l * M * D);
    g->pre.push_back(bf(i_pre) + (int64_t)l * M * Mh);
    g->gact.push_back(bf(i_g) + (int64_t)l * M * Mh);
  }
  g->ucls = bf(i_ucls); g->logits = fl(i_logits); g->dlog = bf(i_dlog); g->ducls = bf(i_ducls);
  g->rowloss = fl(i_rowloss); g->dX = fl(i_dX); g->dXb = bf(i_dXb); g->du = bf(i_du);
  g->dh = bf(i_dh); g->dout = bf(i_dout); g->dqkv = bf(i_dqkv); g->TA = bf(i_TA); g->TB = bf(i_TB);
  g->WT = bf(i_WT); g->WhT = bf(i_WhT); g->part = fl(i_part); g->grad = fl(i_grad);
  g->sq = fl(i_sq); g->stats = fl(i_stats); g->astats = fl(i_astats);

  hipError_t e = hipSuccess;
  uint8_t* sp = at(i_slices);
  for (size_t k = 0; k < host_slices.size() && e == hipSuccess; ++k) {
    g->plans[k].slices = reinterpret_cast<GrowthSlice*>(sp);
    const int64_t bytes = (int64_t)host_slices[k].size() * sizeof(GrowthSlice);
    if (bytes > 0) e = hipMemcpy(sp, host_slices[k].data(), (size_t)bytes, hipMemcpyHostToDevice);
    sp += al256(bytes);
  }
  // Masters of the re-trainable matrices.
  for (int l = 0; l < L && e == hipSuccess; ++l)
    for (int id : {ELASTO_T_WQKV, ELASTO_T_WO, ELASTO_T_W1, ELASTO_T_W2}) {
      const TensorSpec ts = h->lay.get(id, l);
      e = launch_master_init(h->dw, ts.offset / 2, ts.rows * ts.cols, g->master, nullptr);
      if (e != hipSuccess) break;
    }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    (void)hipFree(g->mem);
    delete g;
    return fail(ELASTO_ERR_HIP, "growth set-up: %s", hipGetErrorString(e));
  }
  *out = g;
  clear_error();
  return ELASTO_OK;
}

elasto_status_t elasto_growth_destroy(elasto_growth_t g) {
  if (!g) return ELASTO_OK;
  int cur = -1;
  if (hipGetDevice(&cur) == hipSuccess && cur != g->device) (void)hipSetDevice(g->device);
  if (g->mem) (void)hipFree(g->mem);
  delete g;
  return ELASTO_OK;
}

elasto_status_t elasto_growth_read(elasto_growth_t g, int32_t which, void* host_dst, int64_t bytes) {
  if (!g || !host_dst) return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  const int64_t want = which == 0 ? g->h->lay.total : which == 1 ? g->h->lay.total / 2 * 4 : -1;
  if (want < 0) return fail(ELASTO_ERR_INVALID_ARG, "which must be 0 or 1");
  if (bytes != want) return fail(ELASTO_ERR_INVALID_ARG, "bytes %lld != %lld", (long long)bytes, (long long)want);
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != g->h->device) {
    if (hipSetDevice(g->h->device) != hipSuccess) return fail(ELASTO_ERR_HIP, "cannot select device");
  }
  const void* src = which == 0 ? static_cast<const void*>(g->h->dw) : static_cast<const void*>(g->master);
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(host_dst, src, (size_t)bytes, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "growth read: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

elasto_status_t elasto_growth_step(elasto_growth_t g, int32_t mode, const void* images,
                                   const int32_t* labels, int32_t batch, float lr,
                                   float clip_norm, float* stats, void* hip_stream) {
  if (!g) return fail(ELASTO_ERR_INVALID_ARG, "context is NULL");
  elasto_handle_s* h = g->h;
  if (!images || !labels) return fail(ELASTO_ERR_INVALID_ARG, "images / labels is NULL");
  if (batch < 1 || batch > g->max_batch)
    return fail(ELASTO_ERR_BATCH_RANGE, "batch %d outside [1, %d]", batch, g->max_batch);
  if (mode < 0 || mode + 1 >= h->num_modes)
    return fail(ELASTO_ERR_MODE_RANGE, "mode %d has no smaller mode to grow from", mode);
  const char* why = nullptr;
  if (!growable(h, mode, &why)) return fail(ELASTO_ERR_BAD_TABLE, "%s", why);
  if (!isfinite(lr) || !(clip_norm > 0.0f)) return fail(ELASTO_ERR_INVALID_ARG, "lr must be finite, clip_norm > 0");
  if (!aligned(images, 16) || !aligned(labels, 4) || (stats && !aligned(stats, 4)))
    return fail(ELASTO_ERR_INVALID_ARG, "misaligned pointer");
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
    if (hipSetDevice(h->device) != hipSuccess) return fail(ELASTO_ERR_HIP, "cannot select device %d", h->device);
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const elasto_config_t& c = h->cfg;
  const Dims& d = h->dims;
  const int L = c.depth, D = c.dim, Mh = c.mlp_hidden, C = c.num_classes, T = d.T;
  const int64_t M = (int64_t)batch * T, Mp8 = g->Mp8;
  const ModePlan& plan = g->plans[mode];
  const float scale = 1.0f / sqrtf((float)d.hd);
  hipError_t e = hipSuccess;
#define G_TRY(call, what, ...)                                                                   \
  do {                                                                                          \
    e = (call);                                                                                 \
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, what ": %s", ##__VA_ARGS__, hipGetErrorString(e)); \
  } while (0)

  auto gemm = [&](Epi epi, const void* A, int64_t lda, const void* W, int64_t ldw, void* Cp,
                  int64_t ldc, const float* bias, int64_t rows, int N, int K) {
    GemmArgs a;
    a.A = A; a.lda = lda; a.W = W; a.ldw = ldw; a.C = Cp; a.ldc = ldc; a.bias = bias;
    a.M = rows; a.N = N; a.K = K;
    return a;
  };
  // Weight gradient out[r][c] = sum_m At[r][m] * Bt[c][m] (At: ra rows, Bt: rb
  // rows, both [.][Mp8] bf16) into the gradient arena (row stride rb).
  auto wgrad = [&](const uint16_t* At, int ra, const uint16_t* Bt, int rb, float* outp) {
    if (ra <= 0 || rb <= 0) return hipSuccess;
    const int64_t tiles = ((ra + 255) / 256) * (int64_t)((rb + 255) / 256);
    const int64_t ksteps = (M + 63) / 64;
    int split = (int)std::min<int64_t>({32, std::max<int64_t>(1, 512 / tiles), std::max<int64_t>(1, ksteps / 4)});
    const int64_t kchunk = ((ksteps + split - 1) / split) * 64;
    split = (int)((M + kchunk - 1) / kchunk);
    const int64_t ldp = up4(rb);
    GemmArgs a = gemm(Epi::BiasF32, At, Mp8, Bt, Mp8, g->part, ldp, nullptr, ra, rb, (int)M);
    a.ksplit = split;
    a.kchunk = (int)kchunk;
    a.c_split = (int64_t)ra * ldp;
    if (split > 1 && a.c_split * split > g->part_floats) return hipErrorInvalidValue;
    if (split == 1) a.ksplit = 1;
    hipError_t r = launch_gemm_bf16(Epi::BiasF32, a, s);
    if (r != hipSuccess) return r;
    return launch_splitk_reduce(g->part, a.c_split, split, ra, rb, ldp, outp, rb, s);
  };

  // ------------------------------------------------------------ forward
  {
    GemmArgs a = gemm(Epi::Patch, nullptr, 0, Wb(h, ELASTO_T_PATCH_W), d.patch_k, g->X[0], D,
                      Fp(h, ELASTO_T_PATCH_B), M, D, d.patch_k);
    a.img = images; a.img_size = c.img; a.patch = c.patch; a.chans = c.in_chans; a.grid = d.grid;
    a.tokens = T; a.cls = Fp(h, ELASTO_T_CLS); a.pos = Fp(h, ELASTO_T_POS); a.ldpos = D;
    G_TRY(launch_gemm_bf16(Epi::Patch, a, s), "patch embedding");
  }
  for (int l = 0; l < L; ++l) {
    const LayerPlan& lp = plan.layers[l];
    G_TRY(launch_layernorm_bf16(g->X[l], D, nullptr, T, g->u1[l], M, D, Fp(h, ELASTO_T_LN1_G, l),
                                Fp(h, ELASTO_T_LN1_B, l), c.ln_eps, s), "ln1 layer %d", l);
    G_TRY(launch_gemm_bf16(Epi::Bias, gemm(Epi::Bias, g->u1[l], D, Wb(h, ELASTO_T_WQKV, l), D,
                                           g->qkv[l], 3 * D, Fp(h, ELASTO_T_BQKV, l), M, 192 * lp.h, D), s),
          "qkv layer %d", l);
    AttnArgs at;
    at.qkv = g->qkv[l]; at.qkv_stride = 3 * D; at.o = g->o[l]; at.o_stride = D;
    at.batch = batch; at.tokens = T; at.heads = lp.h; at.head_dim = 64; at.scale = scale;
    G_TRY(launch_attention_bf16(at, s), "attention layer %d", l);
    {
      GemmArgs a = gemm(Epi::BiasResid, g->o[l], D, Wb(h, ELASTO_T_WO, l), D, g->Xm[l], D,
                        Fp(h, ELASTO_T_BO, l), M, D, 64 * lp.h);
      a.res = g->X[l]; a.ldres = D;
      G_TRY(launch_gemm_bf16(Epi::BiasResid, a, s), "proj layer %d", l);
    }
    G_TRY(launch_layernorm_bf16(g->Xm[l], D, nullptr, T, g->u2[l], M, D, Fp(h, ELASTO_T_LN2_G, l),
                                Fp(h, ELASTO_T_LN2_B, l), c.ln_eps, s), "ln2 layer %d", l);
    {
      GemmArgs a = gemm(Epi::BiasGelu, g->u2[l], D, Wb(h, ELASTO_T_W1, l), D, g->gact[l], Mh,
                        Fp(h, ELASTO_T_B1, l), M, lp.m, D);
      a.aux = g->pre[l]; a.ldaux = Mh;
      G_TRY(launch_gemm_bf16(Epi::BiasGelu, a, s), "fc1 layer %d", l);
    }
    {
      GemmArgs a = gemm(Epi::BiasResid, g->gact[l], Mh, Wb(h, ELASTO_T_W2, l), Mh, g->X[l + 1], D,
                        Fp(h, ELASTO_T_B2, l), M, D, lp.m);
      a.res = g->Xm[l]; a.ldres = D;
      G_TRY(launch_gemm_bf16(Epi::BiasResid, a, s), "fc2 layer %d", l);
    }
  }
  G_TRY(launch_layernorm_bf16(g->X[L], (int64_t)T * D, nullptr, 1, g->ucls, batch, D,
                              Fp(h, ELASTO_T_NORM_G), Fp(h, ELASTO_T_NORM_B), c.ln_eps, s), "final norm");
  G_TRY(launch_gemm_bf16(Epi::BiasF32, gemm(Epi::BiasF32, g->ucls, D, Wb(h, ELASTO_T_HEAD_W), D,
                                            g->logits, g->ldlogits, Fp(h, ELASTO_T_HEAD_B), batch, C, D), s),
        "head");

  // ------------------------------------------------------------ backward
  G_TRY(launch_cross_entropy(g->logits, g->ldlogits, labels, C, batch, g->dlog, g->ldlog,
                             g->rowloss, s), "cross-entropy");
  G_TRY(launch_transpose_bf16(Wb(h, ELASTO_T_HEAD_W), D, 0, C, D, g->WhT, g->ldlog, s), "head^T");
  G_TRY(launch_gemm_bf16(Epi::Bias, gemm(Epi::Bias, g->dlog, g->ldlog, g->WhT, g->ldlog, g->ducls, D,
                                         nullptr, batch, D, C), s), "head backward");
  G_TRY(hipMemsetAsync(g->dX, 0, (size_t)(M * D * 4), s), "clear dX");
  G_TRY(hipMemsetAsync(g->dXb, 0, (size_t)(M * D * 2), s), "clear dX bf16");
  G_TRY(launch_layernorm_bwd_bf16(g->X[L], (int64_t)T * D, g->ducls, D, Fp(h, ELASTO_T_NORM_G),
                                  c.ln_eps, batch, D, g->dX, (int64_t)T * D, g->dXb, (int64_t)T * D, s),
        "final norm backward");
  for (int l = L - 1; l >= 0; --l) {
    const LayerPlan& lp = plan.layers[l];
    const int dm = lp.m - lp.mp, dhd = lp.h - lp.hp;
    // fc2
    G_TRY(launch_transpose_bf16(Wb(h, ELASTO_T_W2, l), Mh, 0, D, lp.m, g->WT, D, s), "W2^T %d", l);
    {
      GemmArgs a = gemm(Epi::GeluBwd, g->dXb, D, g->WT, D, g->dh, Mh, nullptr, M, lp.m, D);
      a.aux = g->pre[l]; a.ldaux = Mh;
      G_TRY(launch_gemm_bf16(Epi::GeluBwd, a, s), "fc2 backward %d", l);
    }
    if (dm > 0) {
      G_TRY(launch_transpose_bf16(g->dXb, D, 0, (int)M, D, g->TA, Mp8, s), "dX^T %d", l);
      G_TRY(launch_transpose_bf16(g->gact[l], Mh, lp.mp, (int)M, dm, g->TB, Mp8, s), "g^T %d", l);
      G_TRY(wgrad(g->TA, D, g->TB, dm, g->grad + lp.fc2w), "dW2 %d", l);
    }
    // fc1
    G_TRY(launch_transpose_bf16(Wb(h, ELASTO_T_W1, l), D, 0, lp.m, D, g->WT, up8(lp.m), s), "W1^T %d", l);
    G_TRY(launch_gemm_bf16(Epi::Bias, gemm(Epi::Bias, g->dh, Mh, g->WT, up8(lp.m), g->du, D, nullptr,
                                           M, D, lp.m), s), "fc1 backward %d", l);
    if (dm > 0) {
      G_TRY(launch_transpose_bf16(g->dh, Mh, lp.mp, (int)M, dm, g->TB, Mp8, s), "dh^T %d", l);
      G_TRY(launch_transpose_bf16(g->u2[l], D, 0, (int)M, D, g->TA, Mp8, s), "u2^T %d", l);
      G_TRY(wgrad(g->TB, dm, g->TA, D, g->grad + lp.fc1w), "dW1 %d", l);
      G_TRY(launch_rowsum_bf16(g->TB, Mp8, dm, (int)M, g->grad + lp.fc1b, s), "db1 %d", l);
    }
    G_TRY(launch_layernorm_bwd_bf16(g->Xm[l], D, g->du, D, Fp(h, ELASTO_T_LN2_G, l), c.ln_eps,
                                    (int)M, D, g->dX, D, g->dXb, D, s), "ln2 backward %d", l);
    // proj
    G_TRY(launch_transpose_bf16(Wb(h, ELASTO_T_WO, l), D, 0, D, 64 * lp.h, g->WT, D, s), "WO^T %d", l);
    G_TRY(launch_gemm_bf16(Epi::Bias, gemm(Epi::Bias, g->dXb, D, g->WT, D, g->dout, D, nullptr, M,
                                           64 * lp.h, D), s), "proj backward %d", l);
    if (dhd > 0) {
      G_TRY(launch_transpose_bf16(g->dXb, D, 0, (int)M, D, g->TA, Mp8, s), "dX^T %d", l);
      G_TRY(launch_transpose_bf16(g->o[l], D, 64 * lp.hp, (int)M, 64 * dhd, g->TB, Mp8, s), "o^T %d", l);
      G_TRY(wgrad(g->TA, D, g->TB, 64 * dhd, g->grad + lp.proj), "dWO %d", l);
    }
    // attention
    {
      AttnBwdArgs ab;
      ab.qkv = g->qkv[l]; ab.qkv_stride = 3 * D; ab.dout = g->dout; ab.dout_stride = D;
      ab.dqkv = g->dqkv; ab.dqkv_stride = 3 * D; ab.stats = g->astats;
      ab.batch = batch; ab.tokens = T; ab.heads = lp.h; ab.head_dim = 64; ab.scale = scale;
      G_TRY(launch_attention_bwd_bf16(ab, s), "attention backward %d", l);
    }
    // qkv
    G_TRY(launch_transpose_bf16(Wb(h, ELASTO_T_WQKV, l), D, 0, 192 * lp.h, D, g->WT, 192 * lp.h, s),
          "WQKV^T %d", l);
    G_TRY(launch_gemm_bf16(Epi::Bias, gemm(Epi::Bias, g->dqkv, 3 * D, g->WT, 192 * lp.h, g->du, D,
                                           nullptr, M, D, 192 * lp.h), s), "qkv backward %d", l);
    if (dhd > 0) {
      G_TRY(launch_transpose_bf16(g->dqkv, 3 * D, 192 * lp.hp, (int)M, 192 * dhd, g->TB, Mp8, s),
            "dqkv^T %d", l);
      G_TRY(launch_transpose_bf16(g->u1[l], D, 0, (int)M, D, g->TA, Mp8, s), "u1^T %d", l);
      G_TRY(wgrad(g->TB, 192 * dhd, g->TA, D, g->grad + lp.qkvw), "dWQKV %d", l);
      G_TRY(launch_rowsum_bf16(g->TB, Mp8, 192 * dhd, (int)M, g->grad + lp.qkvb, s), "dbqkv %d", l);
    }
    G_TRY(launch_layernorm_bwd_bf16(g->X[l], D, g->du, D, Fp(h, ELASTO_T_LN1_G, l), c.ln_eps,
                                    (int)M, D, g->dX, D, g->dXb, D, s), "ln1 backward %d", l);
  }
  // ------------------------------------------------- clip and update
  G_TRY(launch_growth_norm(g->grad, plan.grad_floats, g->sq, g->rowloss, batch, clip_norm, g->stats, s),
        "gradient norm");
  G_TRY(launch_growth_update(plan.slices, plan.nslices, g->grad, g->master, h->dw, g->stats, lr, s),
        "update");
  // The inference forward reads LayerNorm-folded copies of the q/k/v and fc1
  // weights: bring them up to date with the updated packed weights.
  G_TRY(refold(h, s), "refold");
  if (stats) G_TRY(hipMemcpyAsync(stats, g->stats, 3 * sizeof(float), hipMemcpyDeviceToDevice, s), "stats");
#undef G_TRY
  return ELASTO_OK;
}

}  // extern "C"
