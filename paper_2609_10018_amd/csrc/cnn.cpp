// C ABI of the elastic bottleneck-ResNet path: validation, packing into the
// prefix layout, buffers, and the forward as a sequence of launches.
//
// One forward in mode k (NHWC bf16 activations; n = n_width[k][b]):
//   stem: NCHW images -> zero-bordered NHWC with 4 channels; 7x7 stride-2
//          implicit convolution (each kernel row one 8-pixel window, the
//          8th pixel and 4th channel with zero weights) + ReLU
//   3x3 stride-2 max pool                                       -> cur
//   per bottleneck b:
//     1x1 reduce: GEMM over cur, N = n (prefix of order1) + ReLU -> t1
//     3x3: implicit-GEMM convolution over t1's first n channels (K runs
//          over the 9 taps, each reading the first n entries of its segment
//          of the packed filter row), N = n (order2) + ReLU          -> t2
//     shortcut: cur, or a 1x1 projection (implicit convolution when
//          strided)                                              -> other
//     1x1 expand: GEMM over t2, K = n, + shortcut, ReLU, in place into the
//          shortcut buffer (which becomes cur)
//   global average pool -> classifier GEMM (fp32 logits)
//
// Tile plans and stream split: at create, for max_batch >= kTuneMinBatch,
// every convolution and GEMM of the forward of every mode (a "site") is
// timed with each tile plan that can run it (kernels.h, kTilePlans,
// plans.h) and keeps the fastest, or the planner's own choice unless another
// plan is faster by the margin (plans.h); the same is done for a forward of
// half the images.  Then each mode's full forward is timed against two
// half-batch forwards, the second on a side stream of the handle (images
// are independent, so the halves only fork and join): a kernel's last
// partial round of tiles then overlaps the other half's kernels.  The split
// is kept where it is faster by the margin.  The choices are kept per
// process for handles of the same shapes (plans.h).  None of these GEMMs has LayerNorm work, so every
// plan and the split give bit-identical outputs: the choices change the
// speed only.  Forwards of more than half of max_batch images use them;
// smaller ones run whole with the planner.
#include <hip/hip_runtime.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "kernels.h"
#include "layout.h"
#include "plans.h"

using namespace elasto;

namespace {

struct BlockSpec {
  int c_in, width, c_out, stride, hw_in;
  bool down;
};

struct BlockOff {
  int64_t c1w, c1b, c2w, c2b, c3w, c3b, dnw, dnb;
};


std::vector<BlockSpec> block_specs(const elasto_cnn_config_t& c) {
  std::vector<BlockSpec> out;
  int c_in = c.stem, hw = c.img / 4;
  for (int s = 0; s < c.num_stages; ++s)
    for (int b = 0; b < c.blocks[s]; ++b) {
      BlockSpec k;
      k.c_in = c_in;
      k.width = c.widths[s];
      k.c_out = c.widths[s] * c.expansion;
      k.stride = (b == 0 && s > 0) ? 2 : 1;
      k.hw_in = hw;
      k.down = b == 0;
      out.push_back(k);
      hw /= k.stride;
      c_in = k.c_out;
    }
  return out;
}

int64_t al256(int64_t v) { return (v + 255) / 256 * 256; }

// Packed stem filter row: 7 kernel rows x (8 pixels x 4 channels).
constexpr int kStemLdw = 7 * 32;

// The stem and the max pool run as one kernel for 32 or 64 stem channels
// (launch_stem_pool); other widths take the padded-input convolution and a
// separate pool.
static bool stem_pool_fused(const elasto_cnn_config_t& c) { return c.stem == 32 || c.stem == 64; }

bool check_cnn_config(const elasto_cnn_config_t* c) {
  if (!c) { set_error("config is NULL"); return false; }
  if (c->dtype != ELASTO_BF16) { set_error("the CNN path is bf16 only"); return false; }
  if (c->img < 32 || c->img % 32 != 0) { set_error("img must be a positive multiple of 32"); return false; }
  if (c->in_chans < 1 || c->in_chans > 4) { set_error("in_chans outside [1, 4]"); return false; }
  if (c->stem < 8 || c->stem % 8 != 0) { set_error("stem channels must be a multiple of 8"); return false; }
  if (c->num_stages < 1 || c->num_stages > 8) { set_error("num_stages outside [1, 8]"); return false; }
  if (c->expansion < 1 || c->num_classes < 1 || c->max_batch < 1) { set_error("bad size"); return false; }
  if ((c->img >> (c->num_stages + 1)) < 1) { set_error("too many stages for img"); return false; }
  for (int s = 0; s < c->num_stages; ++s) {
    if (c->widths[s] < 8 || c->widths[s] % 8 != 0) { set_error("widths must be multiples of 8"); return false; }
    if (c->blocks[s] < 1) { set_error("every stage needs a block"); return false; }
  }
  return true;
}

bool check_cnn_table(const elasto_cnn_config_t* c, const elasto_cnn_table_t* t) {
  if (!t) { set_error("table is NULL"); return false; }
  const std::vector<BlockSpec> bs = block_specs(*c);
  if (t->num_blocks != (int)bs.size()) { set_error("table has %d blocks, the network %d", t->num_blocks, (int)bs.size()); return false; }
  if (t->num_modes < 1 || t->num_modes > 4096) { set_error("num_modes outside [1, 4096]"); return false; }
  if (!t->n_width || !t->order1 || !t->order2) { set_error("table has a NULL array"); return false; }
  for (int k = 0; k < t->num_modes; ++k)
    for (size_t b = 0; b < bs.size(); ++b) {
      const int n = t->n_width[(size_t)k * bs.size() + b];
      if (n < 8 || n > bs[b].width || n % 8 != 0) {
        set_error("n_width[%d][%d] = %d not a multiple of 8 in [8, %d]", k, (int)b, n, bs[b].width);
        return false;
      }
    }
  int64_t off = 0;
  std::vector<char> seen;
  for (size_t b = 0; b < bs.size(); ++b) {
    for (const int32_t* ord : {t->order1, t->order2}) {
      seen.assign(bs[b].width, 0);
      for (int j = 0; j < bs[b].width; ++j) {
        const int v = ord[off + j];
        if (v < 0 || v >= bs[b].width || seen[v]) { set_error("block %d filter order is not a permutation", (int)b); return false; }
        seen[v] = 1;
      }
    }
    off += bs[b].width;
  }
  return true;
}

int num_tensors(const std::vector<BlockSpec>& bs) {
  int n = 4;  // stem w, b; fc w, b
  for (const BlockSpec& b : bs) n += b.down ? 8 : 6;
  return n;
}

}  // namespace

struct elasto_cnn_s {
  elasto_cnn_config_t cfg;
  std::vector<BlockSpec> blocks;
  int num_modes = 0;
  std::vector<int32_t> n_width;  // [num_modes][blocks]
  int mode = 0, device = 0;
  uint8_t* dw = nullptr;
  uint8_t* ds = nullptr;
  int64_t wbytes = 0, sbytes = 0;
  int64_t stem_w = 0, stem_b = 0, fc_w = 0, fc_b = 0;
  std::vector<BlockOff> boff;
  void *col = nullptr, *stem_out = nullptr, *x = nullptr, *d = nullptr, *t1 = nullptr,
       *t2 = nullptr, *feat = nullptr;
  int64_t sz_io = 0, sz_t1 = 0;
  // Per-image capacity (bf16 elements) of each activation buffer: a forward
  // part starting at image slot s uses the buffer from s * capacity on, its
  // images packed at each stage's own size.
  int64_t per_col = 0, per_stem = 0, per_io = 0, per_t1 = 0, per_t2 = 0, per_feat = 0;
  // Tile plan per (mode, site), sites in forward order: per block reduce,
  // 3x3, projection (if any), expand; then the classifier; for whole
  // forwards and for half-batch ones.  Empty: none.
  int nsites = 0;
  std::vector<uint8_t> plans, plans_half;
  std::vector<uint8_t> split;       // per mode: run as two half-batch forwards
  hipStream_t side = nullptr;       // the second half's stream
  hipEvent_t fork = nullptr, join = nullptr;
};

namespace {
// One part of a forward, launched on one stream with a plan per site, or
// (tuning) recording the timed choices.  Its images occupy the activation
// buffers' image slots from slot0 on, a region no other part touches while
// it runs (the buffers are reused from stage to stage with other per-image
// sizes, so each part keeps to its own slots).
struct CnnPart {
  int64_t slot0 = 0;
  const uint8_t* plans = nullptr;  // [nsites], or nullptr: the planner
  uint8_t* tune = nullptr;         // [nsites]: time every plan and record
  hipEvent_t e0 = nullptr, e1 = nullptr;
};
elasto_status_t cnn_run(elasto_cnn_t h, const void* images, int32_t batch, float* logits,
                        hipStream_t s, const CnnPart& part);
elasto_status_t cnn_forward(elasto_cnn_t h, const void* images, int32_t batch, float* logits,
                            hipStream_t s);
void release(elasto_cnn_t h) {
  if (h->side) (void)hipStreamDestroy(h->side);
  if (h->fork) (void)hipEventDestroy(h->fork);
  if (h->join) (void)hipEventDestroy(h->join);
}
}

extern "C" {

elasto_status_t elasto_cnn_validate(const elasto_cnn_config_t* cfg, const elasto_cnn_table_t* t) {
  if (!cfg || !t) return fail(ELASTO_ERR_INVALID_ARG, "%s is NULL", cfg ? "DN table" : "config");
  if (!check_cnn_config(cfg)) return ELASTO_ERR_BAD_CONFIG;
  if (!check_cnn_table(cfg, t)) return ELASTO_ERR_BAD_TABLE;
  clear_error();
  return ELASTO_OK;
}

elasto_status_t elasto_cnn_create(const elasto_cnn_config_t* cfg, const elasto_cnn_weights_t* w,
                                  const elasto_cnn_table_t* table, elasto_cnn_t* out) {
  if (!out || !cfg || !table)
    return fail(ELASTO_ERR_INVALID_ARG, "%s is NULL", !out ? "out" : !cfg ? "config" : "DN table");
  if (!check_cnn_config(cfg)) return ELASTO_ERR_BAD_CONFIG;
  if (!check_cnn_table(cfg, table)) return ELASTO_ERR_BAD_TABLE;
  const std::vector<BlockSpec> bs = block_specs(*cfg);
  if (!w || !w->tensors || w->num_tensors != num_tensors(bs))
    return fail(ELASTO_ERR_INVALID_ARG, "expected %d weight tensors", num_tensors(bs));
  for (int i = 0; i < w->num_tensors; ++i)
    if (!w->tensors[i]) return fail(ELASTO_ERR_INVALID_ARG, "weight tensor %d is NULL", i);

  elasto_cnn_s* h = new (std::nothrow) elasto_cnn_s();
  if (!h) return fail(ELASTO_ERR_OUT_OF_MEMORY, "host allocation failed");
  h->cfg = *cfg;
  h->blocks = bs;
  h->num_modes = table->num_modes;
  h->n_width.assign(table->n_width, table->n_width + (size_t)table->num_modes * bs.size());

  // Packed layout (offsets in bytes, 256-aligned): bf16 filters, fp32 biases.
  const int C = cfg->in_chans;

  int64_t off = 0;
  auto put = [&](int64_t bytes) { const int64_t o = off; off = al256(off + bytes); return o; };
  h->stem_w = put((int64_t)cfg->stem * kStemLdw * 2);
  h->stem_b = put((int64_t)cfg->stem * 4);
  for (const BlockSpec& b : bs) {
    BlockOff o{};
    o.c1w = put((int64_t)b.width * b.c_in * 2);
    o.c1b = put((int64_t)b.width * 4);
    o.c2w = put((int64_t)b.width * b.width * 9 * 2);
    o.c2b = put((int64_t)b.width * 4);
    o.c3w = put((int64_t)b.c_out * b.width * 2);
    o.c3b = put((int64_t)b.c_out * 4);
    if (b.down) {
      o.dnw = put((int64_t)b.c_out * b.c_in * 2);
      o.dnb = put((int64_t)b.c_out * 4);
    }
    h->boff.push_back(o);
  }
  const int F = bs.back().c_out;
  h->fc_w = put((int64_t)cfg->num_classes * F * 2);
  h->fc_b = put((int64_t)cfg->num_classes * 4);
  h->wbytes = off;

  std::vector<uint8_t> host;
  try {
    host.assign((size_t)h->wbytes, 0);
  } catch (...) {
    delete h;
    return fail(ELASTO_ERR_OUT_OF_MEMORY, "host staging allocation failed");
  }
  auto mat = [&](int64_t o, int64_t i, float v) {
    const uint16_t b16 = f32_to_bf16_rne(v);
    memcpy(host.data() + o + i * 2, &b16, 2);
  };
  auto vec = [&](int64_t o, int64_t i, float v) { memcpy(host.data() + o + i * 4, &v, 4); };
  int ti = 0;
  const float* const* T = w->tensors;
  {
    const float* sw = T[ti++];
    const float* sb = T[ti++];
    for (int co = 0; co < cfg->stem; ++co) {
      // [co][i*32 + j*4 + c]: kernel row i, column j < 7, channel c < C; the
      // rest (j == 7, c >= C) stays zero.
      for (int c = 0; c < C; ++c)
        for (int i = 0; i < 7; ++i)
          for (int j = 0; j < 7; ++j)
            mat(h->stem_w, (int64_t)co * kStemLdw + i * 32 + j * 4 + c,
                sw[(((int64_t)co * C + c) * 7 + i) * 7 + j]);
      vec(h->stem_b, co, sb[co]);
    }
  }
  int64_t ooff = 0;
  for (size_t bi = 0; bi < bs.size(); ++bi) {
    const BlockSpec& b = bs[bi];
    const BlockOff& o = h->boff[bi];
    const int32_t* o1 = table->order1 + ooff;
    const int32_t* o2 = table->order2 + ooff;
    ooff += b.width;
    const float *c1w = T[ti], *c1b = T[ti + 1], *c2w = T[ti + 2], *c2b = T[ti + 3],
                *c3w = T[ti + 4], *c3b = T[ti + 5];
    ti += 6;
    for (int j = 0; j < b.width; ++j) {  // reduce: filter j = order1[j]
      for (int c = 0; c < b.c_in; ++c) mat(o.c1w, (int64_t)j * b.c_in + c, c1w[(int64_t)o1[j] * b.c_in + c]);
      vec(o.c1b, j, c1b[o1[j]]);
    }
    for (int j = 0; j < b.width; ++j) {  // 3x3: filter order2[j], tap t, input channel order1[i]
      for (int t = 0; t < 9; ++t)
        for (int i = 0; i < b.width; ++i)
          mat(o.c2w, ((int64_t)j * 9 + t) * b.width + i,
              c2w[(((int64_t)o2[j] * b.width) + o1[i]) * 9 + t]);
      vec(o.c2b, j, c2b[o2[j]]);
    }
    for (int co = 0; co < b.c_out; ++co) {  // expand: input channel order2[i]
      for (int i = 0; i < b.width; ++i) mat(o.c3w, (int64_t)co * b.width + i, c3w[(int64_t)co * b.width + o2[i]]);
      vec(o.c3b, co, c3b[co]);
    }
    if (b.down) {
      const float *dw = T[ti], *db = T[ti + 1];
      ti += 2;
      for (int64_t i = 0; i < (int64_t)b.c_out * b.c_in; ++i) mat(o.dnw, i, dw[i]);
      for (int co = 0; co < b.c_out; ++co) vec(o.dnb, co, db[co]);
    }
  }
  {
    const float* fw = T[ti++];
    const float* fb = T[ti++];
    for (int64_t i = 0; i < (int64_t)cfg->num_classes * F; ++i) mat(h->fc_w, i, fw[i]);
    for (int n = 0; n < cfg->num_classes; ++n) vec(h->fc_b, n, fb[n]);
  }

  // Scratch for max_batch images.
  const int64_t B = cfg->max_batch, hs = cfg->img / 2;
  int64_t col = B * (cfg->img + 6) * (cfg->img + 6) * 4, io = B * (hs / 2) * (hs / 2) * cfg->stem, t1 = 0, t2 = 0;
  for (const BlockSpec& b : bs) {
    const int64_t hi = b.hw_in, ho = b.hw_in / b.stride;
    io = std::max(io, B * ho * ho * b.c_out);
    t1 = std::max(t1, B * hi * hi * b.width);
    t2 = std::max(t2, B * ho * ho * b.width);
  }
  // The fused stem + max pool (32 or 64 stem channels) needs neither the
  // padded NHWC input nor the full-resolution stem output.
  const bool fused = stem_pool_fused(*cfg);
  const int64_t sz_col = fused ? 0 : al256(col * 2),
                sz_stem = fused ? 0 : al256(B * hs * hs * cfg->stem * 2),
                sz_io = al256(io * 2), sz_t1 = al256(t1 * 2), sz_t2 = al256(t2 * 2),
                sz_feat = al256(B * F * 2);
  h->sbytes = sz_col + sz_stem + 2 * sz_io + sz_t1 + sz_t2 + sz_feat;

  hipError_t e = hipGetDevice(&h->device);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&h->dw), (size_t)h->wbytes);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&h->ds), (size_t)h->sbytes);
  if (e == hipSuccess) e = hipMemcpy(h->dw, host.data(), (size_t)h->wbytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    const elasto_status_t st = (e == hipErrorOutOfMemory) ? ELASTO_ERR_OUT_OF_MEMORY : ELASTO_ERR_HIP;
    if (h->dw) (void)hipFree(h->dw);
    if (h->ds) (void)hipFree(h->ds);
    delete h;
    (void)hipGetLastError();
    return fail(st, "cnn create: %s", hipGetErrorString(e));
  }
  uint8_t* p = h->ds;
  h->col = p; p += sz_col;
  h->stem_out = p; p += sz_stem;
  h->x = p; p += sz_io;
  h->d = p; p += sz_io;
  h->t1 = p; p += sz_t1;
  h->t2 = p; p += sz_t2;
  h->feat = p;
  h->sz_io = sz_io;
  h->sz_t1 = sz_t1;
  h->per_col = fused ? 0 : col / B;
  h->per_stem = fused ? 0 : hs * hs * cfg->stem;
  h->per_io = io / B;
  h->per_t1 = t1 / B;
  h->per_t2 = t2 / B;
  h->per_feat = F;
  h->nsites = 1;
  for (const BlockSpec& b : bs) h->nsites += b.down ? 4 : 3;

  // Tile plans and split (file comment): the tuning forwards read their
  // images from the projection buffer d (overwritten only after the stem
  // has read them) and write their logits to t1 (free by then); their values
  // do not matter.
  if (B >= kTuneMinBatch && B * C * cfg->img * cfg->img * 2 <= sz_io &&
      B * cfg->num_classes * 4 <= sz_t1) {
    elasto_status_t st = ELASTO_OK;
    std::vector<int64_t> key;
    bool cached = false;
    try {
      key = {1, h->device, cfg->img, cfg->in_chans, cfg->stem, cfg->num_stages, cfg->expansion,
             cfg->num_classes, cfg->max_batch, cfg->dtype, h->num_modes};
      for (int i = 0; i < cfg->num_stages; ++i) {
        key.push_back(cfg->widths[i]);
        key.push_back(cfg->blocks[i]);
      }
      key.insert(key.end(), h->n_width.begin(), h->n_width.end());
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
      }
    } catch (...) {
      st = fail(ELASTO_ERR_OUT_OF_MEMORY, "host allocation failed");
    }
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (st == ELASTO_OK &&
        (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess ||
         hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) != hipSuccess ||
         hipEventCreateWithFlags(&h->fork, hipEventDisableTiming) != hipSuccess ||
         hipEventCreateWithFlags(&h->join, hipEventDisableTiming) != hipSuccess))
      st = fail(ELASTO_ERR_HIP, "cnn create: cannot create streams / events");
    const void* img = h->d;
    float* lg = static_cast<float*>(h->t1);
    const int32_t Bi = (int32_t)B;
    // Whole forwards and two-stream splits of the mode, alternately (the
    // first pass untimed), and whether the split is faster by the margin.
    auto choose_split = [&](size_t m) -> elasto_status_t {
      float t[2] = {0.0f, 0.0f};
      for (int r = 0; r <= kTuneReps; ++r)
        for (int sp = 0; sp < 2; ++sp) {
          h->split[m] = (uint8_t)sp;
          if (hipEventRecord(e0, nullptr) != hipSuccess) return fail(ELASTO_ERR_HIP, "cnn create: event");
          const elasto_status_t fs = cnn_forward(h, img, Bi, lg, nullptr);
          if (fs != ELASTO_OK) return fs;
          float ms = 0.0f;
          if (hipEventRecord(e1, nullptr) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
              hipEventElapsedTime(&ms, e0, e1) != hipSuccess)
            return fail(ELASTO_ERR_HIP, "cnn create: timing failed");
          if (r == 1 || (r > 1 && ms < t[sp])) t[sp] = ms;
        }
      h->split[m] = t[1] < kTuneMargin * t[0] ? 1 : 0;
      return ELASTO_OK;
    };
    for (int m = 0; st == ELASTO_OK && !cached && m < h->num_modes; ++m) {
      h->mode = m;
      const size_t o = (size_t)m * h->nsites;
      CnnPart full, half;
      full.tune = h->plans.data() + o;
      half.tune = h->plans_half.data() + o;
      full.e0 = half.e0 = e0;
      full.e1 = half.e1 = e1;
      st = cnn_run(h, img, Bi, lg, nullptr, full);
      if (st == ELASTO_OK) st = cnn_run(h, img, Bi / 2, lg, nullptr, half);
      if (st == ELASTO_OK) st = choose_split((size_t)m);
    }
    if (st == ELASTO_OK && hipDeviceSynchronize() != hipSuccess)
      st = fail(ELASTO_ERR_HIP, "cnn create: tuning forward failed");
    if (st == ELASTO_OK && !cached) {
      try {
        tuned_store(key, TunedPlans{h->plans, h->plans_half, h->split});
      } catch (...) {
        st = fail(ELASTO_ERR_OUT_OF_MEMORY, "host allocation failed");
      }
    }
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    h->mode = 0;
    if (st != ELASTO_OK) {
      release(h);
      (void)hipFree(h->dw);
      (void)hipFree(h->ds);
      delete h;
      return st;
    }
  }
  *out = h;
  clear_error();
  return ELASTO_OK;
}

elasto_status_t elasto_cnn_destroy(elasto_cnn_t h) {
  if (!h) return ELASTO_OK;
  hipError_t e1 = hipSuccess, e2 = hipSuccess;
  release(h);
  if (h->dw) e1 = hipFree(h->dw);
  if (h->ds) e2 = hipFree(h->ds);
  delete h;
  if (e1 != hipSuccess || e2 != hipSuccess)
    return fail(ELASTO_ERR_HIP, "cnn destroy: %s", hipGetErrorString(e1 != hipSuccess ? e1 : e2));
  return ELASTO_OK;
}

elasto_status_t elasto_cnn_set_mode(elasto_cnn_t h, int32_t k) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (k < 0 || k >= h->num_modes) return fail(ELASTO_ERR_MODE_RANGE, "mode %d outside [0, %d)", k, h->num_modes);
  h->mode = k;
  return ELASTO_OK;
}

elasto_status_t elasto_cnn_get_mode(elasto_cnn_t h, int32_t* k) {
  if (!h || !k) return fail(ELASTO_ERR_INVALID_ARG, "NULL argument");
  *k = h->mode;
  return ELASTO_OK;
}

elasto_status_t elasto_cnn_mode_info(elasto_cnn_t h, int32_t k, double* macs_per_image,
                                     int64_t* active_weight_bytes) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (k < 0 || k >= h->num_modes) return fail(ELASTO_ERR_MODE_RANGE, "mode %d outside [0, %d)", k, h->num_modes);
  const elasto_cnn_config_t& c = h->cfg;
  const int64_t hs = c.img / 2;
  double macs = (double)hs * hs * c.stem * c.in_chans * 49;
  int64_t wb = (int64_t)c.stem * c.in_chans * 49;
  for (size_t b = 0; b < h->blocks.size(); ++b) {
    const BlockSpec& s = h->blocks[b];
    const int64_t n = h->n_width[(size_t)k * h->blocks.size() + b];
    const double hi = s.hw_in, ho = s.hw_in / s.stride;
    macs += hi * hi * n * s.c_in + ho * ho * n * n * 9 + ho * ho * s.c_out * n;
    wb += n * s.c_in + n * n * 9 + (int64_t)s.c_out * n;
    if (s.down) {
      macs += ho * ho * s.c_out * s.c_in;
      wb += (int64_t)s.c_out * s.c_in;
    }
  }
  macs += (double)h->blocks.back().c_out * c.num_classes;
  wb += (int64_t)h->blocks.back().c_out * c.num_classes;
  if (macs_per_image) *macs_per_image = macs;
  if (active_weight_bytes) *active_weight_bytes = wb * 2;
  return ELASTO_OK;
}

elasto_status_t elasto_cnn_forward(elasto_cnn_t h, const void* images, int32_t batch,
                                   float* logits, void* hip_stream) {
  if (!h) return fail(ELASTO_ERR_INVALID_ARG, "handle is NULL");
  if (!images || !logits) return fail(ELASTO_ERR_INVALID_ARG, "images / logits is NULL");
  if (batch < 1 || batch > h->cfg.max_batch)
    return fail(ELASTO_ERR_BATCH_RANGE, "batch %d outside [1, %d]", batch, h->cfg.max_batch);
  if ((reinterpret_cast<uintptr_t>(images) & 15) != 0 || (reinterpret_cast<uintptr_t>(logits) & 3) != 0)
    return fail(ELASTO_ERR_INVALID_ARG, "misaligned images / logits");
  int cur_dev = -1;
  if (hipGetDevice(&cur_dev) != hipSuccess || cur_dev != h->device) {
    if (hipSetDevice(h->device) != hipSuccess) return fail(ELASTO_ERR_HIP, "cannot select device %d", h->device);
  }
  return cnn_forward(h, images, batch, logits, static_cast<hipStream_t>(hip_stream));
}

}  // extern "C"

namespace {
// A forward of more than half of max_batch images with the tuned plans,
// whole or (split) as two halves, the second on the side stream; smaller
// batches whole with the planner.
elasto_status_t cnn_forward(elasto_cnn_t h, const void* images, int32_t batch, float* logits,
                            hipStream_t s) {
  const elasto_cnn_config_t& c = h->cfg;
  const int k = h->mode;
  const bool tuned = !h->plans.empty() && 2 * (int64_t)batch > c.max_batch;
  CnnPart whole;
  if (!tuned) return cnn_run(h, images, batch, logits, s, whole);
  const size_t o = (size_t)k * h->nsites;
  if (!h->split[(size_t)k]) {
    whole.plans = h->plans.data() + o;
    return cnn_run(h, images, batch, logits, s, whole);
  }
  // The first part takes ceil(batch / 2) images in slots [0, ceil(max_batch / 2)),
  // the second the rest from slot ceil(max_batch / 2) on.
  const int32_t b1 = (batch + 1) / 2, b2 = batch - b1;
  CnnPart first, second;
  first.plans = second.plans = h->plans_half.data() + o;
  second.slot0 = (c.max_batch + 1) / 2;
  if (hipEventRecord(h->fork, s) != hipSuccess || hipStreamWaitEvent(h->side, h->fork, 0) != hipSuccess)
    return fail(ELASTO_ERR_HIP, "cnn forward: cannot fork to the side stream");
  elasto_status_t st = cnn_run(h, images, b1, logits, s, first);
  const elasto_status_t st2 = cnn_run(
      h, static_cast<const uint8_t*>(images) + (int64_t)b1 * c.in_chans * c.img * c.img * 2, b2,
      logits + (int64_t)b1 * c.num_classes, h->side, second);
  if (st == ELASTO_OK) st = st2;
  // Join even after an error, so that the caller's stream orders after both halves.
  if (hipEventRecord(h->join, h->side) != hipSuccess || hipStreamWaitEvent(s, h->join, 0) != hipSuccess)
    return fail(ELASTO_ERR_HIP, "cnn forward: cannot join the side stream");
  return st;
}

// One forward of `batch` images (the file comment) as part `part` of the
// caller's batch; tuning parts time every tile plan at each site and record
// the choices.
elasto_status_t cnn_run(elasto_cnn_t h, const void* images, int32_t batch, float* logits,
                        hipStream_t s, const CnnPart& part) {
  const elasto_cnn_config_t& c = h->cfg;
  const int k = h->mode;
  const int64_t B = batch;
  auto Wp = [&](int64_t o) { return static_cast<const void*>(h->dw + o); };
  auto Fp = [&](int64_t o) { return reinterpret_cast<const float*>(h->dw + o); };
  // Where the part's region starts in an activation buffer of `per` bf16
  // elements of capacity per image (its images are packed from there).
  auto act = [&](void* buf, int64_t per) {
    return static_cast<void*>(static_cast<uint8_t*>(buf) + part.slot0 * per * 2);
  };
  auto gemm = [&](Epi epi, const void* A, int64_t lda, int64_t wo, int64_t ldw, void* C, int64_t ldc,
                  int64_t bo, int64_t M, int N, int K, bool relu, int plan) {
    GemmArgs a;
    a.A = A; a.lda = lda;
    a.W = Wp(wo); a.ldw = ldw;
    a.C = C; a.ldc = ldc;
    a.bias = Fp(bo);
    a.M = M; a.N = N; a.K = K;
    a.relu = relu;
    a.plan = plan;
    return launch_gemm_bf16(epi, a, s);
  };
  // Square input (hw x hw, channel stride cs, first ca channels), ks x ks taps.
  auto conv = [&](const void* x, int hw, int cs, int ca, int ks, int stride, int pad, int64_t wo,
                  int64_t ldw, int64_t wseg, void* C, int64_t ldc, int64_t bo, int N, bool relu,
                  int plan) {
    ConvArgs a;
    a.x = x; a.batch = batch; a.H = hw; a.W = hw; a.Cs = cs; a.Ca = ca;
    a.KH = ks; a.KW = ks; a.stride = stride; a.pad = pad;
    a.weight = Wp(wo); a.ldw = ldw; a.wseg = wseg;
    a.C = C; a.ldc = ldc;
    a.bias = Fp(bo);
    a.N = N;
    a.relu = relu;
    a.plan = plan;
    return launch_conv_bf16(a, s);
  };
  // Site: launch(plan) with the part's plan for the next site, or (tuning)
  // every plan, timed.
  int site = 0;
  auto at_site = [&](auto&& launch) -> hipError_t {
    const int i = site++;
    if (part.tune) return time_plans(launch, s, part.e0, part.e1, &part.tune[i]);
    return launch(part.plans ? (int)part.plans[i] : 0);
  };
  hipError_t e;
#define ELASTO_TRY(call, what)                                                       \
  do {                                                                              \
    e = (call);                                                                     \
    if (e != hipSuccess) return fail(ELASTO_ERR_HIP, "%s: %s", what, hipGetErrorString(e)); \
  } while (0)

  const int hs = c.img / 2;
  if (stem_pool_fused(c)) {
    ELASTO_TRY(launch_stem_pool(images, batch, c.in_chans, c.img, Wp(h->stem_w), kStemLdw,
                                Fp(h->stem_b), c.stem, act(h->x, h->per_io), s),
               "stem + max pool");
  } else {
    void* col = act(h->col, h->per_col);
    void* stem_out = act(h->stem_out, h->per_stem);
    ELASTO_TRY(launch_pad_nhwc4(images, batch, c.in_chans, c.img, c.img, 3, col, s),
               "stem input");
    ConvArgs a;
    a.x = col; a.batch = batch; a.H = c.img + 6; a.W = c.img + 6; a.Cs = 4; a.Ca = 32;
    a.KH = 7; a.KW = 1; a.stride = 2; a.pad = 0; a.row_window = 7;
    a.weight = Wp(h->stem_w); a.ldw = kStemLdw; a.wseg = 32;
    a.C = stem_out; a.ldc = c.stem;
    a.bias = Fp(h->stem_b);
    a.N = c.stem;
    a.relu = true;
    ELASTO_TRY(launch_conv_bf16(a, s), "stem");
    ELASTO_TRY(launch_max_pool_3x3_s2(stem_out, batch, hs, hs, c.stem, act(h->x, h->per_io), s),
               "max pool");
  }
  // Block input and projection output alternate between the x and d buffers.
  void* curb = h->x;
  void* othb = h->d;
  for (size_t bi = 0; bi < h->blocks.size(); ++bi) {
    const BlockSpec& b = h->blocks[bi];
    const BlockOff& o = h->boff[bi];
    const int n = h->n_width[(size_t)k * h->blocks.size() + bi];
    const int hi = b.hw_in, ho = b.hw_in / b.stride;
    const int64_t mi = B * hi * hi, mo = B * ho * ho;
    void* cur = act(curb, h->per_io);
    void* t1 = act(h->t1, h->per_t1);
    void* t2 = act(h->t2, h->per_t2);
    ELASTO_TRY(at_site([&](int pl) {
                 return gemm(Epi::Bias, cur, b.c_in, o.c1w, b.c_in, t1, b.width, o.c1b, mi, n,
                             b.c_in, true, pl);
               }), "1x1 reduce");
    ELASTO_TRY(at_site([&](int pl) {
                 return conv(t1, hi, b.width, n, 3, b.stride, 1, o.c2w, 9 * b.width, b.width,
                             t2, b.width, o.c2b, n, true, pl);
               }), "3x3");
    void* shortcut = cur;
    if (b.down) {
      void* other = act(othb, h->per_io);
      ELASTO_TRY(at_site([&](int pl) {
                   return b.stride > 1
                              ? conv(cur, hi, b.c_in, b.c_in, 1, b.stride, 0, o.dnw, b.c_in, b.c_in,
                                     other, b.c_out, o.dnb, b.c_out, false, pl)
                              : gemm(Epi::Bias, cur, b.c_in, o.dnw, b.c_in, other, b.c_out, o.dnb,
                                     mo, b.c_out, b.c_in, false, pl);
                 }), "projection");
      shortcut = other;
    }
    ELASTO_TRY(at_site([&](int pl) {
                 return gemm(Epi::BiasResid, t2, b.width, o.c3w, b.width, shortcut, b.c_out,
                             o.c3b, mo, b.c_out, n, true, pl);
               }), "1x1 expand");
    if (b.down) std::swap(curb, othb);
  }
  const BlockSpec& last = h->blocks.back();
  const int hf = last.hw_in / last.stride;
  void* feat = act(h->feat, h->per_feat);
  ELASTO_TRY(launch_avg_pool(act(curb, h->per_io), batch, hf * hf, last.c_out, feat, s),
             "average pool");
  ELASTO_TRY(at_site([&](int pl) {
               return gemm(Epi::BiasF32, feat, last.c_out, h->fc_w, last.c_out, logits,
                           c.num_classes, h->fc_b, B, c.num_classes, last.c_out, false, pl);
             }), "classifier");
#undef ELASTO_TRY
  return ELASTO_OK;
}
}  // namespace
