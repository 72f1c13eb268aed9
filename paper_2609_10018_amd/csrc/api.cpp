// C ABI: handle lifecycle, mode switch, forward enqueue, kernel timing and
// the single-kernel entry points.
//
// One forward in mode k on `batch` images (M = batch * tokens rows):
//   patch GEMM (+bias, +pos; class rows = cls + pos[0])          -> x
//   per layer l, with h = n_heads[k][l], m = n_mlp[k][l]:
//     LN1(x)                                                     -> u
//     q/k/v GEMM, N = 3*hd*h (prefix rows of WQKV)               -> qkv
//     attention over h head slots                                -> o
//     projection GEMM, K = hd*h (prefix of each WO row), + x     -> x
//     LN2(x)                                                     -> u
//     fc1 GEMM + GELU, N = m (prefix rows of W1)                 -> g
//     fc2 GEMM, K = m (prefix of each W2 row), + x               -> x
//   final LN on the class rows                                   -> ucls
//   classifier GEMM (fp32 out)                                   -> logits
// Nothing is allocated or synchronised here; the mode is read at enqueue.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "handle.h"
#include "kernels.h"
#include "layout.h"
#include "plans.h"

using namespace elasto;

namespace {

const void* W(const elasto_handle_s* h, int id, int layer = 0) {
  return h->dw + h->lay.get(id, layer).offset;
}
const float* F(const elasto_handle_s* h, int id, int layer = 0) {
  return reinterpret_cast<const float*>(W(h, id, layer));
}

void destroy_events(elasto_handle_s* h) {
  for (hipEvent_t e : h->events) (void)hipEventDestroy(e);
  h->events.clear();
  h->used = 0;
  h->skipped = 0;
  h->timed_class = -1;
}

template <class Fn>
hipError_t timed(elasto_handle_s* h, int kc, hipStream_t s, Fn&& fn) {
  if (kc != h->timed_class) return fn();
  if ((size_t)(2 * h->used + 1) >= h->events.size()) {
    ++h->skipped;
    return fn();
  }
  hipError_t e = hipEventRecord(h->events[2 * h->used], s);
  if (e != hipSuccess) return e;
  e = fn();
  if (e != hipSuccess) return e;
  e = hipEventRecord(h->events[2 * h->used + 1], s);
  ++h->used;
  return e;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

void release_streams(elasto_handle_s* h) {
  if (h->side) (void)hipStreamDestroy(h->side);
  if (h->fork) (void)hipEventDestroy(h->fork);
  if (h->join) (void)hipEventDestroy(h->join);
  h->side = nullptr;
  h->fork = h->join = nullptr;
}

// Activation buffers of one forward.
struct Acts {
  void *x = nullptr, *u = nullptr, *o = nullptr, *qkv = nullptr, *g = nullptr, *ucls = nullptr;
  float* xcls = nullptr;
  float2* lnpart = nullptr;
  float* ws = nullptr;
  int64_t ws_bytes = 0;
};

// Carves the activation buffers of a forward of up to `batch` images out of
// `base` (nullptr: sizes only) and returns the bytes they take.  x is the
// residual stream and u, o, qkv, g, ucls hold activations, all in the path's
// dtype; on the bf16 path the class-token rows of the residual stream are
// kept in fp32 in xcls (they alone decide the logits) and lnpart holds the
// per-segment LayerNorm statistics of every row of x (lnseg float2 a row);
// ws_bytes more (a multiple of 256) follow for the split-K workspace of the
// small-batch GEMMs.
int64_t scratch_layout(const elasto_config_t& cfg, const Dims& d, int lnseg, int64_t batch,
                       int64_t ws_bytes, uint8_t* base, Acts* a) {
  const int64_t eb = cfg.dtype == ELASTO_BF16 ? 2 : 4;
  const int64_t rows = batch * d.T, D = cfg.dim;
  auto al = [](int64_t v) { return (v + 255) / 256 * 256; };
  const int64_t sz_x = al(rows * D * eb), sz_qkv = al(rows * 3 * D * eb),
                sz_g = al(rows * (int64_t)cfg.mlp_hidden * eb), sz_cls = al(batch * D * eb),
                sz_xcls = al(batch * D * 4), sz_ln = lnseg > 0 ? al(rows * lnseg * 8) : 0;
  if (base && a) {
    uint8_t* p = base;
    a->x = p; p += sz_x;
    a->u = p; p += sz_x;
    a->o = p; p += sz_x;
    a->qkv = p; p += sz_qkv;
    a->g = p; p += sz_g;
    a->ucls = p; p += sz_cls;
    a->xcls = reinterpret_cast<float*>(p); p += sz_xcls;
    a->lnpart = lnseg > 0 ? reinterpret_cast<float2*>(p) : nullptr;
    p += sz_ln;
    a->ws = ws_bytes > 0 ? reinterpret_cast<float*>(p) : nullptr;
    a->ws_bytes = ws_bytes;
  }
  return 3 * sz_x + sz_qkv + sz_g + sz_cls + sz_xcls + sz_ln + ws_bytes;
}

// Create-time tuning of the GEMM tile plans (plans.h): events for the
// timings, where the choices of the forward being tuned go ([nsites]), and
// the plan chosen for each GEMM shape already timed (the layers of a mode,
// and often several modes, share shapes).
struct PlanTuning {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  uint8_t* target = nullptr;
  struct Seen {
    int64_t key[9];
    uint8_t plan;
  };
  std::vector<Seen> seen;
};

// One forward over the activation buffers `act`, with a tile plan per GEMM
// site (`plans`, [nsites]; nullptr: the planner), or timing them (`tune`).
elasto_status_t forward_impl(elasto_handle_t h, const void* images, int32_t batch, float* logits,
                             void* hip_stream, const Acts& act, const uint8_t* plans,
                             PlanTuning* tune = nullptr);

// A forward as the handle's tuning chose for the current mode: for more than
// max_batch / 2 images with its tile plans, whole or as two halves on the
// caller's stream and the side stream; smaller batches (and forwards whose
// kernel launches are being timed) whole with the planner.
elasto_status_t forward_parts(elasto_handle_t h, const void* images, int32_t batch, float* logits,
                              void* hip_stream, const Acts& act);

}  // namespace

// LayerNorm folding (bf16 path).  The q/k/v and fc1 GEMMs read the residual
// stream x itself: with u = (x - mean) * rstd * gamma + beta,
//   u . w = rstd * (x . (gamma (x) w)) - rstd * mean * sum_k gamma_k w_k + beta . w,
// so each LayerNorm's gamma is folded into a copy of the next weights, and
// per embedding width e the column sums of that copy and beta . w (plus the
// bias) are precomputed over the first e channels; the GEMM that writes x
// supplies mean and spread per 64-column segment of every row.
hipError_t refold(elasto_handle_s* h, hipStream_t s) {
  if (!h->dfold) return hipSuccess;
  const elasto_config_t& c = h->cfg;
  const int D = c.dim, M = c.mlp_hidden, nw = (int)h->widths.size();
  constexpr int kChunk = 16;  // widths per fold launch
  for (int l = 0; l < c.depth; ++l) {
    uint8_t* f = h->dfold + (int64_t)l * h->fold_stride;
    for (int w0 = 0; w0 < nw; w0 += kChunk) {
      const int n = std::min(kChunk, nw - w0);
      hipError_t e = launch_ln_fold(
          h->dw + h->lay.get(ELASTO_T_WQKV, l).offset, 3 * D, D,
          reinterpret_cast<const float*>(h->dw + h->lay.get(ELASTO_T_LN1_G, l).offset),
          reinterpret_cast<const float*>(h->dw + h->lay.get(ELASTO_T_LN1_B, l).offset),
          reinterpret_cast<const float*>(h->dw + h->lay.get(ELASTO_T_BQKV, l).offset),
          h->widths.data() + w0, n, f + h->fold_wq,
          reinterpret_cast<float*>(f + h->fold_sq) + (int64_t)w0 * 3 * D,
          reinterpret_cast<float*>(f + h->fold_cq) + (int64_t)w0 * 3 * D, 3 * D, s);
      if (e == hipSuccess)
        e = launch_ln_fold(
            h->dw + h->lay.get(ELASTO_T_W1, l).offset, M, D,
            reinterpret_cast<const float*>(h->dw + h->lay.get(ELASTO_T_LN2_G, l).offset),
            reinterpret_cast<const float*>(h->dw + h->lay.get(ELASTO_T_LN2_B, l).offset),
            reinterpret_cast<const float*>(h->dw + h->lay.get(ELASTO_T_B1, l).offset),
            h->widths.data() + w0, n, f + h->fold_w1,
            reinterpret_cast<float*>(f + h->fold_s1) + (int64_t)w0 * M,
            reinterpret_cast<float*>(f + h->fold_c1) + (int64_t)w0 * M, M, s);
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

extern "C" {

elasto_status_t elasto_create(const elasto_config_t* cfg, const elasto_weights_t* w,
                              const elasto_dn_table_t* table, elasto_handle_t* out) {
  if (!out || !cfg || !table)
    return fail(ELASTO_ERR_INVALID_ARG, "%s is NULL", !out ? "out" : !cfg ? "config" : "DN table");
  if (!check_config(cfg)) return ELASTO_ERR_BAD_CONFIG;
  if (!check_table(cfg, table)) return ELASTO_ERR_BAD_TABLE;
  if (!check_weights(w)) return ELASTO_ERR_INVALID_ARG;

  elasto_handle_s* h = new (std::nothrow) elasto_handle_s();
  if (!h) return fail(ELASTO_ERR_OUT_OF_MEMORY, "host allocation failed");
  h->cfg = *cfg;
  h->dims = dims_of(*cfg);
  h->lay = make_layout(*cfg);
  h->num_modes = table->num_modes;
  const size_t nk = (size_t)table->num_modes * cfg->depth;
  h->n_heads.assign(table->n_heads, table->n_heads + nk);
  h->n_mlp.assign(table->n_mlp, table->n_mlp + nk);
  if (table->n_embed)
    h->n_embed.assign(table->n_embed, table->n_embed + table->num_modes);
  else
    h->n_embed.assign((size_t)table->num_modes, cfg->dim);

  std::vector<uint8_t> host;
  try {
    host.resize((size_t)h->lay.total);
  } catch (...) {
    delete h;
    return fail(ELASTO_ERR_OUT_OF_MEMORY, "host staging allocation failed");
  }
  pack(*cfg, *w, *table, h->lay, host.data());

  const int64_t D = cfg->dim;
  auto al = [](int64_t v) { return (v + 255) / 256 * 256; };
  const bool bf = cfg->dtype == ELASTO_BF16;
  h->lnseg = bf ? (int)((D + 127) / 128 * 2) : 0;  // 64-column segments, rounded up to even
  const int64_t ws_bytes = bf ? kSplitWsBytes : 0;
  h->sbytes = scratch_layout(*cfg, h->dims, h->lnseg, cfg->max_batch, ws_bytes, nullptr, nullptr);
  h->wbytes = h->lay.total;
  if (bf) {
    h->width_idx.resize((size_t)table->num_modes);
    for (int k = 0; k < table->num_modes; ++k) {
      const int32_t wv = h->n_embed[(size_t)k];
      size_t i = 0;
      while (i < h->widths.size() && h->widths[i] != wv) ++i;
      if (i == h->widths.size()) h->widths.push_back(wv);
      h->width_idx[(size_t)k] = (int32_t)i;
    }
    const int64_t nw = (int64_t)h->widths.size(), M = cfg->mlp_hidden;
    int64_t off = 0;
    h->fold_wq = off; off = al(off + 3 * D * D * 2);
    h->fold_w1 = off; off = al(off + M * D * 2);
    h->fold_sq = off; off = al(off + nw * 3 * D * 4);
    h->fold_cq = off; off = al(off + nw * 3 * D * 4);
    h->fold_s1 = off; off = al(off + nw * M * 4);
    h->fold_c1 = off; off = al(off + nw * M * 4);
    h->fold_stride = off;
    h->fold_bytes = off * cfg->depth;
  }

  hipError_t e = hipGetDevice(&h->device);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&h->dw), (size_t)h->wbytes);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&h->ds), (size_t)h->sbytes);
  if (e == hipSuccess && h->fold_bytes > 0)
    e = hipMalloc(reinterpret_cast<void**>(&h->dfold), (size_t)h->fold_bytes);
  if (e == hipSuccess) e = hipMemcpy(h->dw, host.data(), (size_t)h->wbytes, hipMemcpyHostToDevice);
  if (e == hipSuccess && h->dfold) e = refold(h, nullptr);
  if (e == hipSuccess && h->dfold) e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) {
    const elasto_status_t st = (e == hipErrorOutOfMemory) ? ELASTO_ERR_OUT_OF_MEMORY : ELASTO_ERR_HIP;
    if (h->dw) (void)hipFree(h->dw);
    if (h->ds) (void)hipFree(h->ds);
    if (h->dfold) (void)hipFree(h->dfold);
    delete h;
    (void)hipGetLastError();
    return fail(st, "create: %s", hipGetErrorString(e));
  }
  Acts a;
  scratch_layout(*cfg, h->dims, h->lnseg, cfg->max_batch, ws_bytes, h->ds, &a);
  h->x = a.x;
  h->u = a.u;
  h->o = a.o;
  h->qkv = a.qkv;
  h->g = a.g;
  h->ucls = a.ucls;
  h->xcls = a.xcls;
  h->lnpart = a.lnpart;
  h->ws = a.ws;
  h->ws_bytes = a.ws_bytes;
  h->nsites = 2 + 4 * cfg->depth;

  // Tile plans and split (handle.h, plans.h): per mode a tuning forward of
  // max_batch images and one of half as many, then the whole forward timed
  // against the two-stream split; or the choices an earlier handle of the
  // same shapes made in this process.  Images are read from the q/k/v buffer
  // (overwritten only after the patch embedding has read them) and logits
  // written to the fc1 buffer; their values do not matter.
  const int64_t B = cfg->max_batch;
  const int64_t img_bytes = B * cfg->in_chans * cfg->img * cfg->img * 2;
  const int64_t qkv_bytes = B * h->dims.T * 3 * (int64_t)cfg->dim * 2;
  const int64_t g_bytes = B * h->dims.T * (int64_t)cfg->mlp_hidden * 2;
  if (bf && img_bytes <= qkv_bytes && B * cfg->num_classes * 4 <= g_bytes) {
    elasto_status_t st = ELASTO_OK;
    PlanTuning tn;
    std::vector<int64_t> key;
    bool cached = false;
    try {
      key = {0, h->device, cfg->img, cfg->patch, cfg->in_chans, cfg->dim, cfg->depth, cfg->heads,
             cfg->mlp_hidden, cfg->num_classes, cfg->max_batch, cfg->dtype, h->num_modes};
      key.insert(key.end(), h->n_heads.begin(), h->n_heads.end());
      key.insert(key.end(), h->n_mlp.begin(), h->n_mlp.end());
      key.insert(key.end(), h->n_embed.begin(), h->n_embed.end());
      TunedPlans tp;
      cached = tuned_lookup(key, &tp);
      if (cached) {
        h->plans = tp.plans;
        h->plans_half = tp.plans_half;
        h->split = tp.split;
      } else {
        h->plans.assign((size_t)h->num_modes * h->nsites, 0);
        h->plans_half.assign((size_t)h->num_modes * h->nsites, 0);
        h->split.assign((size_t)h->num_modes, 0);
        tn.seen.reserve(64);
      }
    } catch (...) {
      st = fail(ELASTO_ERR_OUT_OF_MEMORY, "host allocation failed");
    }
    if (st == ELASTO_OK &&
        (hipEventCreate(&tn.e0) != hipSuccess || hipEventCreate(&tn.e1) != hipSuccess ||
         hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) != hipSuccess ||
         hipEventCreateWithFlags(&h->fork, hipEventDisableTiming) != hipSuccess ||
         hipEventCreateWithFlags(&h->join, hipEventDisableTiming) != hipSuccess))
      st = fail(ELASTO_ERR_HIP, "create: cannot create streams / events");
    Acts half = a;
    half.ws = nullptr;
    half.ws_bytes = 0;
    float* lg = static_cast<float*>(h->g);
    // Whole forwards and two-stream splits of the mode, alternately (the
    // first pass untimed), and whether the split is faster by the margin.
    auto choose_split = [&](size_t m) -> elasto_status_t {
      float t[2] = {0.0f, 0.0f};
      for (int r = 0; r <= kTuneReps; ++r)
        for (int sp = 0; sp < 2; ++sp) {
          h->split[m] = (uint8_t)sp;
          if (hipEventRecord(tn.e0, nullptr) != hipSuccess) return fail(ELASTO_ERR_HIP, "create: event");
          const elasto_status_t fs = forward_parts(h, h->qkv, (int32_t)B, lg, nullptr, a);
          if (fs != ELASTO_OK) return fs;
          float ms = 0.0f;
          if (hipEventRecord(tn.e1, nullptr) != hipSuccess || hipEventSynchronize(tn.e1) != hipSuccess ||
              hipEventElapsedTime(&ms, tn.e0, tn.e1) != hipSuccess)
            return fail(ELASTO_ERR_HIP, "create: timing failed");
          if (r == 1 || (r > 1 && ms < t[sp])) t[sp] = ms;
        }
      h->split[m] = t[1] < kTuneMargin * t[0] ? 1 : 0;
      return ELASTO_OK;
    };
    for (int m = 0; st == ELASTO_OK && !cached && m < h->num_modes; ++m) {
      h->mode = m;
      const size_t o = (size_t)m * h->nsites;
      tn.target = h->plans.data() + o;
      st = forward_impl(h, h->qkv, (int32_t)B, lg, nullptr, a, nullptr, &tn);
      tn.target = h->plans_half.data() + o;
      if (st == ELASTO_OK)
        st = forward_impl(h, h->qkv, (int32_t)((B + 1) / 2), lg, nullptr, half, nullptr, &tn);
      if (st == ELASTO_OK) st = choose_split((size_t)m);
    }
    if (st == ELASTO_OK && hipDeviceSynchronize() != hipSuccess)
      st = fail(ELASTO_ERR_HIP, "create: tuning forward failed");
    if (st == ELASTO_OK && !cached) {
      try {
        tuned_store(key, TunedPlans{h->plans, h->plans_half, h->split});
      } catch (...) {
        st = fail(ELASTO_ERR_OUT_OF_MEMORY, "host allocation failed");
      }
    }
    if (tn.e0) (void)hipEventDestroy(tn.e0);
    if (tn.e1) (void)hipEventDestroy(tn.e1);
    h->mode = 0;
    if (st != ELASTO_OK) {
      release_streams(h);
      (void)hipFree(h->dw);
      (void)hipFree(h->ds);
      if (h->dfold) (void)hipFree(h->dfold);
      delete h;
      return st;
    }
  }
  *out = h;
  clear_error();
  return ELASTO_OK;
}

elasto_status_t elasto_destroy(elasto_handle_t h) {
  if (!h) return ELASTO_OK;
  destroy_events(h);
  release_streams(h);
  hipError_t e1 = hipSuccess, e2 = hipSuccess;
  if (h->dw) e1 = hipFree(h->dw);
  if (h->ds) e2 = hipFree(h->ds);
  if (h->dfold) {
    const hipError_t e3 = hipFree(h->dfold);
    if (e1 == hipSuccess) e1 = e3;
  }
  delete h;
  if (e1 != hipSuccess || e2 != hipSuccess)
    return fail(ELASTO_ERR_HIP, "destroy: %s", hipGetErrorString(e1 != hipSuccess ? e1 : e2));
  return ELASTO_OK;
}

elasto_status_t elasto_set_mode(elasto_handle_t h, int32_t k) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (k < 0 || k >= h->num_modes) return fail(ELASTO_ERR_MODE_RANGE, "mode %d outside [0, %d)", k, h->num_modes);
  h->mode = k;
  return ELASTO_OK;
}

elasto_status_t elasto_get_mode(elasto_handle_t h, int32_t* k) {
  if (!h || !k) return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  *k = h->mode;
  return ELASTO_OK;
}

elasto_status_t elasto_mode_info(elasto_handle_t h, int32_t k, double* flops_per_image,
                                 int64_t* active_weight_bytes) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (k < 0 || k >= h->num_modes) return fail(ELASTO_ERR_MODE_RANGE, "mode %d outside [0, %d)", k, h->num_modes);
  const int32_t* nh = h->n_heads.data() + (size_t)k * h->cfg.depth;
  const int32_t* nm = h->n_mlp.data() + (size_t)k * h->cfg.depth;
  const int de = h->n_embed[k];
  if (flops_per_image) *flops_per_image = mode_flops(h->cfg, nh, nm, de);
  if (active_weight_bytes) *active_weight_bytes = mode_weight_bytes(h->cfg, nh, nm, de);
  return ELASTO_OK;
}

elasto_status_t elasto_memory_info(elasto_handle_t h, int64_t* weight_bytes, int64_t* scratch_bytes) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (weight_bytes) *weight_bytes = h->wbytes + h->fold_bytes;
  if (scratch_bytes) *scratch_bytes = h->sbytes;
  return ELASTO_OK;
}

elasto_status_t elasto_profile_modes(elasto_handle_t h, const void* images, int32_t batch,
                                     float* logits, int32_t warmup, int32_t iters,
                                     void* hip_stream, double* latency_ms, double* memory_bytes,
                                     double* flops) {
  if (!h || !images || !logits || !latency_ms || !memory_bytes || !flops)
    return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  if (batch < 1 || batch > h->cfg.max_batch)
    return fail(ELASTO_ERR_BATCH_RANGE, "batch %d outside [1, %d]", batch, h->cfg.max_batch);
  if (warmup < 0 || iters < 1 || iters > 1000)
    return fail(ELASTO_ERR_INVALID_ARG, "warmup must be >= 0 and iters in [1, 1000]");
  if ((h->cfg.dtype == ELASTO_BF16 && !aligned(images, 16)) || !aligned(images, 4) ||
      !aligned(logits, 4))
    return fail(ELASTO_ERR_INVALID_ARG, "misaligned images / logits");
  const elasto_config_t& c = h->cfg;
  const Dims& d = h->dims;
  const int L = c.depth;
  const int64_t eb = c.dtype == ELASTO_BF16 ? 2 : 4, rows = (int64_t)batch * d.T;
  for (int k = 0; k < h->num_modes; ++k) {
    const int32_t* nh = h->n_heads.data() + (size_t)k * L;
    const int32_t* nm = h->n_mlp.data() + (size_t)k * L;
    const int64_t D = h->n_embed[k];
    int64_t vec = 2 * D + (int64_t)d.T * D + 2 * D + c.num_classes;  // patch_b, cls, pos, norm, head_b
    int64_t hmax = 0, mmax = 0;
    for (int l = 0; l < L; ++l) {
      vec += 2 * D + 3 * d.hd * nh[l] + D + 2 * D + nm[l] + D;  // ln1, bqkv, bo, ln2, b1, b2
      hmax = nh[l] > hmax ? nh[l] : hmax;
      mmax = nm[l] > mmax ? nm[l] : mmax;
    }
    int64_t act = 2 * rows * D * eb                       // residual stream, LN output
                  + rows * 3 * d.hd * hmax * eb            // q/k/v
                  + rows * d.hd * hmax * eb                // attention output
                  + rows * mmax * eb                       // MLP hidden
                  + (int64_t)batch * D * eb;               // final LN rows
    if (c.dtype == ELASTO_BF16) act += (int64_t)batch * D * 4;  // fp32 class-token rows
    memory_bytes[k] = (double)(mode_weight_bytes(c, nh, nm, (int)D) + vec * 4 + act);
    flops[k] = mode_flops(c, nh, nm, (int)D) * batch;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
    if (hipSetDevice(h->device) != hipSuccess) return fail(ELASTO_ERR_HIP, "cannot select device %d", h->device);
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  std::vector<hipEvent_t> ev(iters + 1, nullptr);
  hipError_t e = hipSuccess;
  elasto_status_t fst = ELASTO_OK;  // status of the forwards
  for (auto& x : ev)
    if (e == hipSuccess) e = hipEventCreate(&x);
  const int saved = h->mode;
  std::vector<double> ms(iters);
  for (int k = 0; k < h->num_modes && e == hipSuccess && fst == ELASTO_OK; ++k) {
    h->mode = k;
    for (int i = 0; i < warmup && fst == ELASTO_OK; ++i)
      fst = elasto_forward(h, images, batch, logits, hip_stream);
    for (int i = 0; i < iters && e == hipSuccess && fst == ELASTO_OK; ++i) {
      e = hipEventRecord(ev[i], s);
      if (e == hipSuccess) fst = elasto_forward(h, images, batch, logits, hip_stream);
      if (e == hipSuccess && fst == ELASTO_OK && i == iters - 1) e = hipEventRecord(ev[iters], s);
    }
    if (fst != ELASTO_OK) break;
    if (e == hipSuccess) e = hipEventSynchronize(ev[iters]);
    for (int i = 0; i < iters && e == hipSuccess; ++i) {
      float t = 0.0f;
      e = hipEventElapsedTime(&t, ev[i], ev[i + 1]);
      ms[i] = t;
    }
    if (e == hipSuccess) {
      std::vector<double> sorted(ms);
      std::sort(sorted.begin(), sorted.end());
      latency_ms[k] = iters % 2 ? sorted[iters / 2]
                                : 0.5 * (sorted[iters / 2 - 1] + sorted[iters / 2]);
    }
  }
  h->mode = saved;
  if (fst != ELASTO_OK) (void)hipStreamSynchronize(s);  // drain before the events go
  for (auto x : ev)
    if (x) (void)hipEventDestroy(x);
  if (fst != ELASTO_OK) return fst;  // the forward's own message stays
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "profiling failed: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

elasto_status_t elasto_forward(elasto_handle_t h, const void* images, int32_t batch, float* logits,
                               void* hip_stream) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  Acts a;
  a.x = h->x; a.u = h->u; a.o = h->o; a.qkv = h->qkv; a.g = h->g; a.ucls = h->ucls;
  a.xcls = h->xcls; a.lnpart = h->lnpart; a.ws = h->ws; a.ws_bytes = h->ws_bytes;
  return forward_parts(h, images, batch, logits, hip_stream, a);
}

elasto_status_t elasto_forward_static(elasto_handle_t h, const void* images, int32_t batch,
                                      float* logits, void* hip_stream) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (batch < 1 || batch > h->cfg.max_batch)
    return fail(ELASTO_ERR_BATCH_RANGE, "batch %d outside [1, %d]", batch, h->cfg.max_batch);
  const int64_t need = scratch_layout(h->cfg, h->dims, h->lnseg, batch, 0, nullptr, nullptr);
  if (need > kStaticScratchBytes)
    return fail(ELASTO_ERR_BATCH_RANGE,
                "batch %d needs %lld bytes of activation scratch; the static scratch holds %lld",
                batch, (long long)need, (long long)kStaticScratchBytes);
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
    if (hipSetDevice(h->device) != hipSuccess) return fail(ELASTO_ERR_HIP, "cannot select device %d", h->device);
  }
  void* base = nullptr;
  int64_t have = 0;
  const hipError_t e = static_scratch(&base, &have);
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "static scratch: %s", hipGetErrorString(e));
  // What the activations leave of the array serves as split-K workspace.
  const int64_t ws_bytes = h->cfg.dtype == ELASTO_BF16
                               ? std::min(kSplitWsBytes, (have - need) / 256 * 256) : 0;
  Acts a;
  scratch_layout(h->cfg, h->dims, h->lnseg, batch, ws_bytes, static_cast<uint8_t*>(base), &a);
  return forward_parts(h, images, batch, logits, hip_stream, a);
}

}  // extern "C"

namespace {

// The activation buffers of the images from `b` on (every buffer holds a
// fixed number of bytes per image), without the split-K workspace.
Acts offset_acts(const elasto_handle_s* h, const Acts& a, int64_t b) {
  const elasto_config_t& c = h->cfg;
  const int64_t eb = c.dtype == ELASTO_BF16 ? 2 : 4, T = h->dims.T, D = c.dim;
  auto adv = [&](void* p, int64_t per_image) {
    return p ? static_cast<void*>(static_cast<uint8_t*>(p) + b * per_image) : nullptr;
  };
  Acts r;
  r.x = adv(a.x, T * D * eb);
  r.u = adv(a.u, T * D * eb);
  r.o = adv(a.o, T * D * eb);
  r.qkv = adv(a.qkv, T * 3 * D * eb);
  r.g = adv(a.g, T * c.mlp_hidden * eb);
  r.ucls = adv(a.ucls, D * eb);
  r.xcls = a.xcls ? a.xcls + b * D : nullptr;
  r.lnpart = a.lnpart ? a.lnpart + b * T * h->lnseg : nullptr;
  return r;
}

elasto_status_t forward_parts(elasto_handle_t h, const void* images, int32_t batch, float* logits,
                              void* hip_stream, const Acts& act) {
  const elasto_config_t& c = h->cfg;
  const int k = h->mode;
  if (h->plans.empty() || 2 * (int64_t)batch <= c.max_batch || batch > c.max_batch)
    return forward_impl(h, images, batch, logits, hip_stream, act, nullptr);
  const size_t o = (size_t)k * h->nsites;
  const int32_t b1 = (batch + 1) / 2, b2 = batch - b1;
  const int64_t img_bytes = (int64_t)c.in_chans * c.img * c.img * 2;
  if (!h->split[(size_t)k] || h->timed_class >= 0 || b2 < 1 || (b1 * img_bytes) % 16 != 0 ||
      !images || !logits)
    return forward_impl(h, images, batch, logits, hip_stream, act, h->plans.data() + o);
  // Neither half gets the split-K workspace (they run at once, and each
  // image's arithmetic must not depend on the half it falls in).
  Acts first = act;
  first.ws = nullptr;
  first.ws_bytes = 0;
  const Acts second = offset_acts(h, act, b1);
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (hipEventRecord(h->fork, s) != hipSuccess || hipStreamWaitEvent(h->side, h->fork, 0) != hipSuccess)
    return fail(ELASTO_ERR_HIP, "forward: cannot fork to the side stream");
  const uint8_t* ph = h->plans_half.data() + o;
  elasto_status_t st = forward_impl(h, images, b1, logits, hip_stream, first, ph);
  const elasto_status_t st2 =
      forward_impl(h, static_cast<const uint8_t*>(images) + b1 * img_bytes, b2,
                   logits + (int64_t)b1 * c.num_classes, h->side, second, ph);
  if (st == ELASTO_OK) st = st2;
  // Join even after an error, so that the caller's stream orders after both halves.
  if (hipEventRecord(h->join, h->side) != hipSuccess || hipStreamWaitEvent(s, h->join, 0) != hipSuccess)
    return fail(ELASTO_ERR_HIP, "forward: cannot join the side stream");
  return st;
}

elasto_status_t forward_impl(elasto_handle_t h, const void* images, int32_t batch, float* logits,
                             void* hip_stream, const Acts& act, const uint8_t* plans,
                             PlanTuning* tune) {
  if (!images || !logits) return fail(ELASTO_ERR_INVALID_ARG, "images / logits is NULL");
  if (batch < 1 || batch > h->cfg.max_batch)
    return fail(ELASTO_ERR_BATCH_RANGE, "batch %d outside [1, %d]", batch, h->cfg.max_batch);
  const bool bf = h->cfg.dtype == ELASTO_BF16;
  if (bf && !aligned(images, 16)) return fail(ELASTO_ERR_INVALID_ARG, "images must be 16-byte aligned");
  if (!aligned(images, 4) || !aligned(logits, 4)) return fail(ELASTO_ERR_INVALID_ARG, "misaligned pointer");

  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
    if (hipSetDevice(h->device) != hipSuccess) return fail(ELASTO_ERR_HIP, "cannot select device %d", h->device);
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const elasto_config_t& c = h->cfg;
  const Dims& d = h->dims;
  const int k = h->mode;
  // D: row stride of the residual stream; E: its active channels in mode k
  // (LayerNorm outputs and the class-token rows are stored E wide).
  const int L = c.depth, D = c.dim, E = h->n_embed[k], Mh = c.mlp_hidden;
  const int64_t rows = (int64_t)batch * d.T;
  auto gemm = bf ? launch_gemm_bf16 : launch_gemm_f32;
  auto attn = bf ? launch_attention_bf16 : launch_attention_f32;
  float* xcls = bf ? act.xcls : nullptr;
  // LayerNorm over all rows of the residual stream.
  auto ln = [&](const float* g, const float* b) {
    return bf ? launch_layernorm_bf16(act.x, D, xcls, d.T, act.u, rows, E, g, b, c.ln_eps, s)
              : launch_layernorm_f32(act.x, D, act.u, rows, E, g, b, c.ln_eps, s);
  };
  const float scale = 1.0f / sqrtf((float)d.hd);
  // bf16: LayerNorms folded into the q/k/v and fc1 GEMMs (see refold); the
  // GEMMs that write the residual stream produce its segment statistics.
  const bool fold = h->dfold != nullptr;
  const int wi = fold ? h->width_idx[(size_t)k] : 0;
  auto fold_ptr = [&](int l, int64_t off) { return h->dfold + (int64_t)l * h->fold_stride + off; };
  // GEMM sites (handle.h): the plan of the next site; in the tuning
  // forwards, every plan timed (once per distinct shape) and the choice
  // recorded.
  int site = 0;
  auto run = [&](int kc, Epi epi, GemmArgs& a) -> hipError_t {
    const int i = site++;
    if (tune) {
      const int64_t key[9] = {(int64_t)epi, a.M, a.N, a.K, a.lda, a.ldc, a.ln_in != nullptr,
                              a.ln_out != nullptr, a.ccls != nullptr};
      for (const PlanTuning::Seen& sn : tune->seen)
        if (std::equal(key, key + 9, sn.key)) {
          tune->target[i] = sn.plan;
          return hipSuccess;
        }
      const hipError_t te = time_plans(
          [&](int pl) {
            a.plan = pl;
            return gemm(epi, a, s);
          },
          s, tune->e0, tune->e1, &tune->target[i]);
      PlanTuning::Seen sn;
      std::copy(key, key + 9, sn.key);
      sn.plan = tune->target[i];
      tune->seen.push_back(sn);
      return te;
    }
    a.plan = plans ? (int)plans[i] : 0;
    return timed(h, kc, s, [&] {
      hipError_t ge = gemm(epi, a, s);
      // A split plan chosen with the handle's workspace may not fit a smaller
      // one (the forward in the static scratch): the planner decides there.
      if (ge == hipErrorNotSupported && a.plan >= kSplitPlan0) {
        a.plan = 0;
        ge = gemm(epi, a, s);
      }
      return ge;
    });
  };

  hipError_t e;
  {
    GemmArgs a;
    a.W = W(h, ELASTO_T_PATCH_W);
    a.ldw = d.patch_k;
    a.C = act.x;
    a.ldc = D;
    a.bias = F(h, ELASTO_T_PATCH_B);
    a.M = rows;
    a.N = E;
    a.K = d.patch_k;
    a.img = images;
    a.img_size = c.img;
    a.patch = c.patch;
    a.chans = c.in_chans;
    a.grid = d.grid;
    a.tokens = d.T;
    a.cls = F(h, ELASTO_T_CLS);
    a.pos = F(h, ELASTO_T_POS);
    a.ldpos = D;
    a.ccls = xcls;
    if (fold) {
      a.ln_out = act.lnpart;
      a.ln_ld = h->lnseg;
    }
    e = run(ELASTO_K_PATCH, Epi::Patch, a);
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "patch embedding: %s", hipGetErrorString(e));
  }
  for (int l = 0; l < L; ++l) {
    const int hh = h->n_heads[(size_t)k * L + l], mm = h->n_mlp[(size_t)k * L + l];
    if (!fold) {
      e = timed(h, ELASTO_K_LN, s, [&] { return ln(F(h, ELASTO_T_LN1_G, l), F(h, ELASTO_T_LN1_B, l)); });
      if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "ln1 layer %d: %s", l, hipGetErrorString(e));
    }
    GemmArgs q;
    q.A = act.u; q.lda = E;
    q.W = W(h, ELASTO_T_WQKV, l); q.ldw = D;
    q.C = act.qkv; q.ldc = 3 * D;
    q.bias = F(h, ELASTO_T_BQKV, l);
    q.M = rows; q.N = 3 * d.hd * hh; q.K = E;
    if (fold) {
      q.A = act.x; q.lda = D;
      q.W = fold_ptr(l, h->fold_wq);
      q.bias = reinterpret_cast<const float*>(fold_ptr(l, h->fold_cq)) + (int64_t)wi * 3 * D;
      q.ln_colsum = reinterpret_cast<const float*>(fold_ptr(l, h->fold_sq)) + (int64_t)wi * 3 * D;
      q.ln_in = act.lnpart; q.ln_ld = h->lnseg; q.ln_eps = c.ln_eps;
    }
    q.ws = act.ws; q.ws_bytes = act.ws_bytes;
    e = run(ELASTO_K_QKV, Epi::Bias, q);
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "qkv layer %d: %s", l, hipGetErrorString(e));
    AttnArgs at;
    at.qkv = act.qkv; at.qkv_stride = 3 * D;
    at.o = act.o; at.o_stride = D;
    at.batch = batch; at.tokens = d.T; at.heads = hh; at.head_dim = d.hd; at.scale = scale;
    e = timed(h, ELASTO_K_ATTN, s, [&] { return attn(at, s); });
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "attention layer %d: %s", l, hipGetErrorString(e));
    GemmArgs pr;
    pr.A = act.o; pr.lda = D;
    pr.W = W(h, ELASTO_T_WO, l); pr.ldw = D;
    pr.C = act.x; pr.ldc = D;
    pr.bias = F(h, ELASTO_T_BO, l);
    pr.ccls = xcls;
    pr.tokens = d.T;
    pr.M = rows; pr.N = E; pr.K = d.hd * hh;
    if (fold) {
      pr.ln_out = act.lnpart; pr.ln_ld = h->lnseg;
    }
    pr.ws = act.ws; pr.ws_bytes = act.ws_bytes;
    e = run(ELASTO_K_PROJ, Epi::BiasResid, pr);
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "proj layer %d: %s", l, hipGetErrorString(e));
    if (!fold) {
      e = timed(h, ELASTO_K_LN, s, [&] { return ln(F(h, ELASTO_T_LN2_G, l), F(h, ELASTO_T_LN2_B, l)); });
      if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "ln2 layer %d: %s", l, hipGetErrorString(e));
    }
    GemmArgs f1;
    f1.A = act.u; f1.lda = E;
    f1.W = W(h, ELASTO_T_W1, l); f1.ldw = D;
    f1.C = act.g; f1.ldc = Mh;
    f1.bias = F(h, ELASTO_T_B1, l);
    f1.M = rows; f1.N = mm; f1.K = E;
    if (fold) {
      f1.A = act.x; f1.lda = D;
      f1.W = fold_ptr(l, h->fold_w1);
      f1.bias = reinterpret_cast<const float*>(fold_ptr(l, h->fold_c1)) + (int64_t)wi * Mh;
      f1.ln_colsum = reinterpret_cast<const float*>(fold_ptr(l, h->fold_s1)) + (int64_t)wi * Mh;
      f1.ln_in = act.lnpart; f1.ln_ld = h->lnseg; f1.ln_eps = c.ln_eps;
    }
    f1.ws = act.ws; f1.ws_bytes = act.ws_bytes;
    e = run(ELASTO_K_FC1, Epi::BiasGelu, f1);
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "fc1 layer %d: %s", l, hipGetErrorString(e));
    GemmArgs f2;
    f2.A = act.g; f2.lda = Mh;
    f2.W = W(h, ELASTO_T_W2, l); f2.ldw = Mh;
    f2.C = act.x; f2.ldc = D;
    f2.bias = F(h, ELASTO_T_B2, l);
    f2.ccls = xcls;
    f2.tokens = d.T;
    f2.M = rows; f2.N = E; f2.K = mm;
    if (fold) {
      f2.ln_out = act.lnpart; f2.ln_ld = h->lnseg;
    }
    f2.ws = act.ws; f2.ws_bytes = act.ws_bytes;
    e = run(ELASTO_K_FC2, Epi::BiasResid, f2);
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "fc2 layer %d: %s", l, hipGetErrorString(e));
  }
  // Final norm on the class-token rows only.
  e = timed(h, ELASTO_K_LN, s, [&] {
    return bf ? launch_layernorm_bf16(xcls, E, xcls, 1, act.ucls, batch, E, F(h, ELASTO_T_NORM_G),
                                      F(h, ELASTO_T_NORM_B), c.ln_eps, s)
              : launch_layernorm_f32(act.x, (int64_t)d.T * D, act.ucls, batch, E,
                                     F(h, ELASTO_T_NORM_G), F(h, ELASTO_T_NORM_B), c.ln_eps, s);
  });
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "final norm: %s", hipGetErrorString(e));
  GemmArgs hg;
  hg.A = act.ucls; hg.lda = E;
  hg.W = W(h, ELASTO_T_HEAD_W); hg.ldw = D;
  hg.C = logits; hg.ldc = c.num_classes;
  hg.bias = F(h, ELASTO_T_HEAD_B);
  hg.M = batch; hg.N = c.num_classes; hg.K = E;
  e = run(ELASTO_K_HEAD, Epi::BiasF32, hg);
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "head: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

}  // namespace

extern "C" {

elasto_status_t elasto_kernel_timing(elasto_handle_t h, int32_t kc, int32_t max_launches) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (kc < -1 || kc >= ELASTO_K_COUNT) return fail(ELASTO_ERR_INVALID_ARG, "kernel class %d out of range", kc);
  destroy_events(h);
  if (kc < 0) return ELASTO_OK;
  if (max_launches < 1 || max_launches > (1 << 20))
    return fail(ELASTO_ERR_INVALID_ARG, "max_launches %d outside [1, 2^20]", max_launches);
  h->events.resize((size_t)2 * max_launches, nullptr);
  for (auto& ev : h->events) {
    if (hipEventCreate(&ev) != hipSuccess) {
      ev = nullptr;
      destroy_events(h);
      return fail(ELASTO_ERR_HIP, "hipEventCreate failed");
    }
  }
  h->timed_class = kc;
  return ELASTO_OK;
}

elasto_status_t elasto_kernel_timing_read(elasto_handle_t h, double* total_ms, int64_t* launches) {
  if (!h || !total_ms || !launches) return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  double sum = 0.0;
  for (int i = 0; i < h->used; ++i) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(h->events[2 * i + 1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, h->events[2 * i], h->events[2 * i + 1]);
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "event read: %s", hipGetErrorString(e));
    sum += ms;
  }
  *total_ms = sum;
  *launches = h->used;
  h->used = 0;
  h->skipped = 0;
  return ELASTO_OK;
}

elasto_status_t elasto_kernel_work(elasto_handle_t h, int32_t k, int32_t batch, int32_t kc,
                                   double* flops, double* bytes, int32_t* launches) {
  if (!h || !flops || !bytes || !launches) return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  if (k < 0 || k >= h->num_modes) return fail(ELASTO_ERR_MODE_RANGE, "mode %d outside [0, %d)", k, h->num_modes);
  if (batch < 1) return fail(ELASTO_ERR_BATCH_RANGE, "batch must be >= 1");
  if (kc < 0 || kc >= ELASTO_K_COUNT) return fail(ELASTO_ERR_INVALID_ARG, "kernel class %d out of range", kc);
  const elasto_config_t& c = h->cfg;
  const Dims& d = h->dims;
  const double eb = c.dtype == ELASTO_BF16 ? 2.0 : 4.0;
  // D: active embedding channels of mode k.
  const double B = batch, T = d.T, D = h->n_embed[k], hd = d.hd, Np = (double)d.grid * d.grid;
  const double Mr = B * T;
  double f = 0, by = 0;
  int n = 0;
  switch (kc) {
    case ELASTO_K_PATCH:
      f = 2.0 * B * Np * d.patch_k * D;
      by = (B * c.in_chans * (double)c.img * c.img + D * d.patch_k + Mr * D) * eb;
      n = 1;
      break;
    case ELASTO_K_LN:
      if (h->dfold) {  // pre-norms folded into the GEMMs: the final norm of the class rows
        by = B * D * (4.0 + eb);
        n = 1;
      } else {
        by = 2.0 * c.depth * Mr * D * 2.0 * eb + B * D * (4.0 + eb);
        n = 2 * c.depth + 1;
      }
      break;
    case ELASTO_K_HEAD:
      f = 2.0 * B * c.num_classes * D;
      by = (B * D + (double)c.num_classes * D) * eb + B * c.num_classes * 4.0;
      n = 1;
      break;
    default:
      for (int l = 0; l < c.depth; ++l) {
        const double hh = h->n_heads[(size_t)k * c.depth + l], mm = h->n_mlp[(size_t)k * c.depth + l];
        switch (kc) {
          case ELASTO_K_QKV:
            f += 2.0 * Mr * 3 * hd * hh * D;
            by += (Mr * D + 3 * hd * hh * D + Mr * 3 * hd * hh) * eb;
            break;
          case ELASTO_K_ATTN:
            f += 4.0 * B * hh * T * T * hd;
            by += (Mr * 3 * hd * hh + Mr * hd * hh) * eb;
            break;
          case ELASTO_K_PROJ:
            f += 2.0 * Mr * D * hd * hh;
            by += (Mr * hd * hh + D * hd * hh + 2.0 * Mr * D) * eb;
            break;
          case ELASTO_K_FC1:
            f += 2.0 * Mr * mm * D;
            by += (Mr * D + mm * D + Mr * mm) * eb;
            break;
          case ELASTO_K_FC2:
            f += 2.0 * Mr * D * mm;
            by += (Mr * mm + D * mm + 2.0 * Mr * D) * eb;
            break;
        }
      }
      n = c.depth;
  }
  *flops = f;
  *bytes = by;
  *launches = n;
  return ELASTO_OK;
}

elasto_status_t elasto_op_layernorm(int32_t dtype, const void* x, int64_t x_stride,
                                    const float* x_cls, int32_t tokens, void* out, int64_t rows,
                                    int32_t d, const float* g, const float* b, float eps,
                                    void* hip_stream) {
  if (!x || !out || !g || !b) return fail(ELASTO_ERR_INVALID_ARG, "NULL pointer");
  if (x_cls && (tokens < 1 || dtype != ELASTO_BF16 || !aligned(x_cls, 16)))
    return fail(ELASTO_ERR_INVALID_ARG, "x_cls needs the bf16 path, tokens >= 1, 16-byte alignment");
  if (rows < 0 || d < 1 || d > 2048 || x_stride < d || !(eps > 0.0f))
    return fail(ELASTO_ERR_INVALID_ARG, "bad layernorm sizes");
  hipError_t e;
  if (dtype == ELASTO_BF16) {
    if (d % 8 != 0 || x_stride % 8 != 0 || !aligned(x, 16) || !aligned(out, 16) ||
        !aligned(g, 16) || !aligned(b, 16))
      return fail(ELASTO_ERR_INVALID_ARG, "bf16 layernorm needs d, stride %% 8 == 0 and 16-byte aligned pointers");
    e = launch_layernorm_bf16(x, x_stride, x_cls, tokens, out, rows, d, g, b, eps,
                              static_cast<hipStream_t>(hip_stream));
  } else if (dtype == ELASTO_FP32) {
    e = launch_layernorm_f32(x, x_stride, out, rows, d, g, b, eps, static_cast<hipStream_t>(hip_stream));
  } else {
    return fail(ELASTO_ERR_INVALID_ARG, "bad dtype %d", dtype);
  }
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "layernorm: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

elasto_status_t elasto_op_linear(int32_t dtype, int32_t epilogue, const void* A, int64_t lda,
                                 const void* Wt, int64_t ldw, void* C, int64_t ldc, float* C_cls,
                                 int32_t tokens, const float* bias, int64_t M, int32_t N,
                                 int32_t K, void* hip_stream) {
  if (!A || !Wt || !C || !bias) return fail(ELASTO_ERR_INVALID_ARG, "NULL pointer");
  if (C_cls && (epilogue != ELASTO_EPI_BIAS_RESID || dtype != ELASTO_BF16 || tokens < 1 ||
                !aligned(C_cls, 16) || N % 4 != 0))
    return fail(ELASTO_ERR_INVALID_ARG,
                "C_cls needs the bf16 residual epilogue, tokens >= 1, N %% 4 == 0, 16-byte alignment");
  if (M < 0 || M >= ((int64_t)1 << 31) || N < 1 || K < 1 || lda < K || ldw < K || ldc < N)
    return fail(ELASTO_ERR_INVALID_ARG, "bad linear sizes");
  if (epilogue < ELASTO_EPI_BIAS || epilogue > ELASTO_EPI_BIAS_F32OUT)
    return fail(ELASTO_ERR_INVALID_ARG, "bad epilogue %d", epilogue);
  GemmArgs a;
  a.A = A; a.lda = lda; a.W = Wt; a.ldw = ldw; a.C = C; a.ldc = ldc; a.bias = bias;
  a.M = M; a.N = N; a.K = K;
  a.ccls = C_cls;
  a.tokens = tokens;
  const Epi epi = static_cast<Epi>(epilogue);
  hipError_t e;
  if (dtype == ELASTO_BF16) {
    const int64_t cvec = epilogue == ELASTO_EPI_BIAS_F32OUT ? 4 : 8;
    if (lda % 8 || ldw % 8 || ldc % cvec || !aligned(A, 16) || !aligned(Wt, 16) || !aligned(C, 16) ||
        !aligned(bias, 16))
      return fail(ELASTO_ERR_INVALID_ARG,
                  "bf16 linear needs lda, ldw %% 8 == 0, ldc a multiple of 16 bytes and 16-byte "
                  "aligned A, W, C, bias");
    e = launch_gemm_bf16(epi, a, static_cast<hipStream_t>(hip_stream));
  } else if (dtype == ELASTO_FP32) {
    e = launch_gemm_f32(epi, a, static_cast<hipStream_t>(hip_stream));
  } else {
    return fail(ELASTO_ERR_INVALID_ARG, "bad dtype %d", dtype);
  }
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "linear: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

elasto_status_t elasto_op_linear_ln(int32_t epilogue, const void* A, int64_t lda, const void* Wt,
                                    int64_t ldw, void* C, int64_t ldc, float* C_cls,
                                    int32_t tokens, const float* bias, int64_t M, int32_t N,
                                    int32_t K, float* stats_out, const float* stats_in,
                                    int64_t stats_ld, const float* colsum, float eps,
                                    void* hip_stream) {
  if (!A || !Wt || !C || !bias) return fail(ELASTO_ERR_INVALID_ARG, "NULL pointer");
  if ((stats_out != nullptr) == (stats_in != nullptr))
    return fail(ELASTO_ERR_INVALID_ARG, "exactly one of stats_out, stats_in must be given");
  if (M < 0 || M >= ((int64_t)1 << 31) || N < 1 || K < 1 || lda < K || ldw < K || ldc < N)
    return fail(ELASTO_ERR_INVALID_ARG, "bad linear sizes");
  if (lda % 8 || ldw % 8 || ldc % 8 || !aligned(A, 16) || !aligned(Wt, 16) || !aligned(C, 16) ||
      !aligned(bias, 16))
    return fail(ELASTO_ERR_INVALID_ARG,
                "linear needs lda, ldw, ldc %% 8 == 0 and 16-byte aligned A, W, C, bias");
  const float* st = stats_out ? stats_out : stats_in;
  const int64_t width = stats_out ? N : K;
  if (!aligned(st, 16) || stats_ld % 2 || stats_ld < (width + 63) / 64)
    return fail(ELASTO_ERR_INVALID_ARG, "stats need 16-byte alignment and an even stats_ld >= ceil(width / 64)");
  GemmArgs a;
  a.A = A; a.lda = lda; a.W = Wt; a.ldw = ldw; a.C = C; a.ldc = ldc; a.bias = bias;
  a.M = M; a.N = N; a.K = K;
  a.ln_ld = stats_ld;
  Epi epi;
  if (stats_out) {
    if (epilogue != ELASTO_EPI_BIAS_RESID || N % 8)
      return fail(ELASTO_ERR_INVALID_ARG, "the producer needs the residual epilogue and N %% 8 == 0");
    if (C_cls && (tokens < 1 || !aligned(C_cls, 16)))
      return fail(ELASTO_ERR_INVALID_ARG, "C_cls needs tokens >= 1 and 16-byte alignment");
    a.ccls = C_cls;
    a.tokens = tokens;
    a.ln_out = reinterpret_cast<float2*>(stats_out);
    epi = Epi::BiasResid;
  } else {
    if (epilogue != ELASTO_EPI_BIAS && epilogue != ELASTO_EPI_BIAS_GELU)
      return fail(ELASTO_ERR_INVALID_ARG, "the consumer needs the bias or bias+GELU epilogue");
    if (C_cls) return fail(ELASTO_ERR_INVALID_ARG, "C_cls is for the producer");
    if (!colsum || !aligned(colsum, 16) || !(eps > 0.0f))
      return fail(ELASTO_ERR_INVALID_ARG, "the consumer needs 16-byte aligned colsum and eps > 0");
    a.ln_in = reinterpret_cast<const float2*>(stats_in);
    a.ln_colsum = colsum;
    a.ln_eps = eps;
    epi = static_cast<Epi>(epilogue);
  }
  const hipError_t e = launch_gemm_bf16(epi, a, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "linear_ln: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

elasto_status_t elasto_op_conv2d(const void* x, int32_t batch, int32_t H, int32_t W, int32_t cs,
                                 int32_t ca, int32_t kh, int32_t kw, int32_t stride, int32_t pad,
                                 const void* w, int64_t ldw, int64_t wseg, const float* bias,
                                 void* y, int64_t ldy, int32_t n, int32_t relu, void* hip_stream) {
  if (!x || !w || !bias || !y) return fail(ELASTO_ERR_INVALID_ARG, "NULL pointer");
  if (batch < 0 || H < 1 || W < 1 || kh < 1 || kw < 1 || stride < 1 || pad < 0 || n < 1 ||
      H + 2 * pad < kh || W + 2 * pad < kw)
    return fail(ELASTO_ERR_INVALID_ARG, "bad convolution sizes");
  if (ca < 8 || ca % 8 || cs % 8 || ca > cs || wseg < ca || wseg % 8 || ldw % 8 ||
      ldw < (int64_t)kh * kw * wseg || ldy < n || ldy % 8)
    return fail(ELASTO_ERR_INVALID_ARG,
                "convolution needs cs, ca, wseg, ldw, ldy %% 8 == 0, 8 <= ca <= min(cs, wseg), "
                "ldw >= kh*kw*wseg, ldy >= n");
  if (!aligned(x, 16) || !aligned(w, 16) || !aligned(y, 16) || !aligned(bias, 16))
    return fail(ELASTO_ERR_INVALID_ARG, "convolution needs 16-byte aligned x, w, y, bias");
  const int64_t limit = ((int64_t)1 << 31) - 1;
  if ((int64_t)H * W * cs * 2 > limit || ((int64_t)(n - 1) * ldw + (int64_t)kh * kw * wseg) * 2 > limit)
    return fail(ELASTO_ERR_INVALID_ARG, "one image's input or the read weights exceed 2 GiB");
  const int64_t ho = (H + 2 * pad - kh) / stride + 1, wo = (W + 2 * pad - kw) / stride + 1;
  if ((int64_t)batch * ho * wo >= ((int64_t)1 << 31))
    return fail(ELASTO_ERR_INVALID_ARG, "too many output pixels");
  ConvArgs a;
  a.x = x; a.batch = batch; a.H = H; a.W = W; a.Cs = cs; a.Ca = ca;
  a.KH = kh; a.KW = kw; a.stride = stride; a.pad = pad;
  a.weight = w; a.ldw = ldw; a.wseg = wseg;
  a.C = y; a.ldc = ldy; a.bias = bias; a.N = n; a.relu = relu != 0;
  const hipError_t e = launch_conv_bf16(a, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "conv2d: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

elasto_status_t elasto_op_attention(int32_t dtype, const void* qkv, int64_t qkv_stride, void* o,
                                    int64_t o_stride, int32_t batch, int32_t tokens,
                                    int32_t heads, int32_t head_dim, float scale,
                                    void* hip_stream) {
  if (!qkv || !o) return fail(ELASTO_ERR_INVALID_ARG, "NULL pointer");
  if (batch < 0 || tokens < 1 || heads < 1 || head_dim < 1 || qkv_stride < 3LL * heads * head_dim ||
      o_stride < (int64_t)heads * head_dim)
    return fail(ELASTO_ERR_INVALID_ARG, "bad attention sizes");
  AttnArgs a;
  a.qkv = qkv; a.qkv_stride = qkv_stride; a.o = o; a.o_stride = o_stride;
  a.batch = batch; a.tokens = tokens; a.heads = heads; a.head_dim = head_dim; a.scale = scale;
  hipError_t e;
  if (dtype == ELASTO_BF16) {
    if (head_dim != 64 || tokens > kAttnMaxTokens || qkv_stride % 8 || !aligned(qkv, 16) ||
        o_stride % 4 || !aligned(o, 8) || (int64_t)tokens * o_stride * 2 > INT32_MAX)
      return fail(ELASTO_ERR_INVALID_ARG,
                  "bf16 attention needs head_dim 64, tokens <= %d, aligned qkv and o, o range < 2^31",
                  kAttnMaxTokens);
    e = launch_attention_bf16(a, static_cast<hipStream_t>(hip_stream));
  } else if (dtype == ELASTO_FP32) {
    if (head_dim > 128) return fail(ELASTO_ERR_INVALID_ARG, "fp32 attention needs head_dim <= 128");
    e = launch_attention_f32(a, static_cast<hipStream_t>(hip_stream));
  } else {
    return fail(ELASTO_ERR_INVALID_ARG, "bad dtype %d", dtype);
  }
  if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "attention: %s", hipGetErrorString(e));
  return ELASTO_OK;
}

}  // extern "C"
