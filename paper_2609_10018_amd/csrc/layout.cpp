// Host-only unit: validation, packed prefix layout, packing, error messages.
//
// Packing puts every layer's channels in the order of the DN table (the order
// in which the nested DNs introduce them, Eq. 8), so that mode k's active
// heads / units are the first n_heads[k][l] / n_mlp[k][l] entries:
//   WQKV row s*3hd + t*hd + c  = qkv_w row t*d + head_order[s]*hd + c
//   WO   column s*hd + c       = proj_w column head_order[s]*hd + c
//   W1   row s                 = fc1_w row mlp_order[s]
//   W2   column s              = fc2_w column mlp_order[s]
// and every embedding axis (length d) in embed_order: packed channel j is
// canonical channel embed_order[j] (identity when the table gives none).
// Matrices are stored in the path's dtype (bf16 rounded to nearest even, or
// fp32); biases, norms, class token and positions stay fp32.
#include "layout.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <vector>

namespace elasto {

namespace {
thread_local std::string g_err;
constexpr int64_t kAlign = 256;
int64_t align_up(int64_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
}  // namespace

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
}

void clear_error() { g_err.clear(); }

elasto_status_t fail(elasto_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

Dims dims_of(const elasto_config_t& c) {
  Dims d;
  d.grid = c.img / c.patch;
  d.T = d.grid * d.grid + 1;
  d.hd = c.dim / c.heads;
  d.patch_k = c.in_chans * c.patch * c.patch;
  return d;
}

bool check_config(const elasto_config_t* c) {
  if (!c) { set_error("config is NULL"); return false; }
  if (c->img < 1 || c->patch < 1 || c->in_chans < 1 || c->dim < 1 || c->depth < 1 ||
      c->heads < 1 || c->mlp_hidden < 1 || c->num_classes < 1 || c->max_batch < 1) {
    set_error("every config size must be >= 1");
    return false;
  }
  if (c->dtype != ELASTO_FP32 && c->dtype != ELASTO_BF16) {
    set_error("dtype %d is neither ELASTO_FP32 nor ELASTO_BF16", c->dtype);
    return false;
  }
  if (!(c->ln_eps > 0.0f) || !isfinite(c->ln_eps)) { set_error("ln_eps must be finite and > 0"); return false; }
  if (c->img % c->patch != 0) { set_error("img %d is not a multiple of patch %d", c->img, c->patch); return false; }
  if (c->dim % c->heads != 0) { set_error("dim %d is not a multiple of heads %d", c->dim, c->heads); return false; }
  if (c->dim > 2048) { set_error("dim %d > 2048 is not supported", c->dim); return false; }
  const Dims d = dims_of(*c);
  if ((int64_t)c->max_batch * d.T * (int64_t)(3 * c->dim > c->mlp_hidden ? 3 * c->dim : c->mlp_hidden) >
      ((int64_t)1 << 40)) {
    set_error("max_batch too large");
    return false;
  }
  if ((int64_t)c->max_batch * d.T >= ((int64_t)1 << 31)) { set_error("max_batch * tokens must be < 2^31"); return false; }
  if (c->dtype == ELASTO_BF16) {
    if (d.hd != 64) { set_error("bf16 path needs head_dim 64 (got %d)", d.hd); return false; }
    if (c->patch % 8 != 0) { set_error("bf16 path needs patch %% 8 == 0"); return false; }
    if (c->dim % 8 != 0 || c->mlp_hidden % 8 != 0) {
      set_error("bf16 path needs dim and mlp_hidden multiples of 8");
      return false;
    }
    if (d.T > 240) { set_error("bf16 path supports at most 240 tokens (got %d)", d.T); return false; }
  } else {
    if (d.hd > 128) { set_error("fp32 path needs head_dim <= 128 (got %d)", d.hd); return false; }
  }
  return true;
}

bool check_table(const elasto_config_t* c, const elasto_dn_table_t* t) {
  if (!t) { set_error("DN table is NULL"); return false; }
  if (t->depth != c->depth) { set_error("table depth %d != config depth %d", t->depth, c->depth); return false; }
  if (t->num_modes < 1 || t->num_modes > 4096) { set_error("num_modes %d outside [1, 4096]", t->num_modes); return false; }
  if (!t->n_heads || !t->n_mlp || !t->head_order || !t->mlp_order) {
    set_error("DN table has a NULL array");
    return false;
  }
  for (int k = 0; k < t->num_modes; ++k)
    for (int l = 0; l < t->depth; ++l) {
      const int h = t->n_heads[k * t->depth + l], m = t->n_mlp[k * t->depth + l];
      if (h < 1 || h > c->heads) { set_error("n_heads[%d][%d] = %d outside [1, %d]", k, l, h, c->heads); return false; }
      if (m < 1 || m > c->mlp_hidden) { set_error("n_mlp[%d][%d] = %d outside [1, %d]", k, l, m, c->mlp_hidden); return false; }
    }
  if (t->n_embed) {
    for (int k = 0; k < t->num_modes; ++k) {
      const int e = t->n_embed[k];
      if (e < 1 || e > c->dim) { set_error("n_embed[%d] = %d outside [1, %d]", k, e, c->dim); return false; }
      if (c->dtype == ELASTO_BF16 && e % 8 != 0) { set_error("n_embed[%d] = %d is not a multiple of 8 (bf16)", k, e); return false; }
    }
  }
  std::vector<char> seen;
  if (t->embed_order) {
    seen.assign(c->dim, 0);
    for (int j = 0; j < c->dim; ++j) {
      const int v = t->embed_order[j];
      if (v < 0 || v >= c->dim || seen[v]) { set_error("embed_order is not a permutation"); return false; }
      seen[v] = 1;
    }
  }
  for (int l = 0; l < t->depth; ++l) {
    seen.assign(c->heads, 0);
    for (int s = 0; s < c->heads; ++s) {
      const int v = t->head_order[(int64_t)l * c->heads + s];
      if (v < 0 || v >= c->heads || seen[v]) { set_error("head_order[%d] is not a permutation", l); return false; }
      seen[v] = 1;
    }
    seen.assign(c->mlp_hidden, 0);
    for (int s = 0; s < c->mlp_hidden; ++s) {
      const int v = t->mlp_order[(int64_t)l * c->mlp_hidden + s];
      if (v < 0 || v >= c->mlp_hidden || seen[v]) { set_error("mlp_order[%d] is not a permutation", l); return false; }
      seen[v] = 1;
    }
  }
  return true;
}

bool check_weights(const elasto_weights_t* w) {
  if (!w) { set_error("weights are NULL"); return false; }
  const float* ptrs[] = {w->patch_w, w->patch_b, w->cls, w->pos, w->ln1_g, w->ln1_b, w->qkv_w,
                         w->qkv_b, w->proj_w, w->proj_b, w->ln2_g, w->ln2_b, w->fc1_w, w->fc1_b,
                         w->fc2_w, w->fc2_b, w->norm_g, w->norm_b, w->head_w, w->head_b};
  for (const float* p : ptrs)
    if (!p) { set_error("a weight pointer is NULL"); return false; }
  return true;
}

TensorSpec Layout::get(int tensor, int layer_idx) const {
  if (tensor < ELASTO_T_LN1_G) return global[tensor];
  TensorSpec s = layer[tensor - ELASTO_T_LN1_G];
  s.offset += layer_base + (int64_t)layer_idx * layer_stride;
  return s;
}

Layout make_layout(const elasto_config_t& c) {
  const Dims d = dims_of(c);
  const int me = c.dtype == ELASTO_BF16 ? 2 : 4;
  const int64_t D = c.dim, M = c.mlp_hidden, C = c.num_classes;
  Layout L{};
  int64_t off = 0;
  auto put = [&](TensorSpec& s, int64_t rows, int64_t cols, int eb) {
    s.offset = off;
    s.rows = rows;
    s.cols = cols;
    s.elem_bytes = eb;
    off = align_up(off + rows * cols * eb);
  };
  put(L.global[ELASTO_T_PATCH_W], D, d.patch_k, me);
  put(L.global[ELASTO_T_PATCH_B], 1, D, 4);
  put(L.global[ELASTO_T_CLS], 1, D, 4);
  put(L.global[ELASTO_T_POS], d.T, D, 4);
  put(L.global[ELASTO_T_NORM_G], 1, D, 4);
  put(L.global[ELASTO_T_NORM_B], 1, D, 4);
  put(L.global[ELASTO_T_HEAD_W], C, D, me);
  put(L.global[ELASTO_T_HEAD_B], 1, C, 4);
  L.layer_base = off;
  off = 0;
  const int b = ELASTO_T_LN1_G;
  put(L.layer[ELASTO_T_LN1_G - b], 1, D, 4);
  put(L.layer[ELASTO_T_LN1_B - b], 1, D, 4);
  put(L.layer[ELASTO_T_WQKV - b], 3 * D, D, me);
  put(L.layer[ELASTO_T_BQKV - b], 1, 3 * D, 4);
  put(L.layer[ELASTO_T_WO - b], D, D, me);
  put(L.layer[ELASTO_T_BO - b], 1, D, 4);
  put(L.layer[ELASTO_T_LN2_G - b], 1, D, 4);
  put(L.layer[ELASTO_T_LN2_B - b], 1, D, 4);
  put(L.layer[ELASTO_T_W1 - b], M, D, me);
  put(L.layer[ELASTO_T_B1 - b], 1, M, 4);
  put(L.layer[ELASTO_T_W2 - b], D, M, me);
  put(L.layer[ELASTO_T_B2 - b], 1, D, 4);
  L.layer_stride = off;
  L.total = L.layer_base + L.layer_stride * c.depth;
  return L;
}

namespace {

struct Writer {
  uint8_t* base;
  bool bf16;
  void mat(int64_t off, int64_t idx, float v) const {
    if (bf16) {
      const uint16_t h = f32_to_bf16_rne(v);
      memcpy(base + off + idx * 2, &h, 2);
    } else {
      memcpy(base + off + idx * 4, &v, 4);
    }
  }
  void vec(int64_t off, int64_t idx, float v) const { memcpy(base + off + idx * 4, &v, 4); }
};

}  // namespace

void pack(const elasto_config_t& c, const elasto_weights_t& w, const elasto_dn_table_t& t,
          const Layout& L, uint8_t* dst) {
  memset(dst, 0, (size_t)L.total);
  const Dims d = dims_of(c);
  const int64_t D = c.dim, M = c.mlp_hidden, C = c.num_classes, H = c.heads, hd = d.hd;
  const Writer wr{dst, c.dtype == ELASTO_BF16};
  // ev[j]: canonical embedding channel stored at packed position j.
  std::vector<int64_t> ev(D);
  for (int64_t j = 0; j < D; ++j) ev[j] = t.embed_order ? t.embed_order[j] : j;
  auto g = [&](int id) { return L.get(id, 0).offset; };
  for (int64_t j = 0; j < D; ++j) {
    for (int64_t k = 0; k < d.patch_k; ++k)
      wr.mat(g(ELASTO_T_PATCH_W), j * d.patch_k + k, w.patch_w[ev[j] * d.patch_k + k]);
    wr.vec(g(ELASTO_T_PATCH_B), j, w.patch_b[ev[j]]);
    wr.vec(g(ELASTO_T_CLS), j, w.cls[ev[j]]);
    wr.vec(g(ELASTO_T_NORM_G), j, w.norm_g[ev[j]]);
    wr.vec(g(ELASTO_T_NORM_B), j, w.norm_b[ev[j]]);
  }
  for (int64_t tk = 0; tk < d.T; ++tk)
    for (int64_t j = 0; j < D; ++j) wr.vec(g(ELASTO_T_POS), tk * D + j, w.pos[tk * D + ev[j]]);
  for (int64_t n = 0; n < C; ++n)
    for (int64_t j = 0; j < D; ++j) wr.mat(g(ELASTO_T_HEAD_W), n * D + j, w.head_w[n * D + ev[j]]);
  for (int64_t i = 0; i < C; ++i) wr.vec(g(ELASTO_T_HEAD_B), i, w.head_b[i]);

  for (int l = 0; l < c.depth; ++l) {
    auto o = [&](int id) { return L.get(id, l).offset; };
    const int32_t* ho = t.head_order + (int64_t)l * H;
    const int32_t* mo = t.mlp_order + (int64_t)l * M;
    for (int64_t j = 0; j < D; ++j) {
      const int64_t i = ev[j];
      wr.vec(o(ELASTO_T_LN1_G), j, w.ln1_g[l * D + i]);
      wr.vec(o(ELASTO_T_LN1_B), j, w.ln1_b[l * D + i]);
      wr.vec(o(ELASTO_T_LN2_G), j, w.ln2_g[l * D + i]);
      wr.vec(o(ELASTO_T_LN2_B), j, w.ln2_b[l * D + i]);
      wr.vec(o(ELASTO_T_BO), j, w.proj_b[l * D + i]);
      wr.vec(o(ELASTO_T_B2), j, w.fc2_b[l * D + i]);
    }
    const float* qkv_w = w.qkv_w + (int64_t)l * 3 * D * D;
    const float* qkv_b = w.qkv_b + (int64_t)l * 3 * D;
    for (int64_t s = 0; s < H; ++s)
      for (int64_t tq = 0; tq < 3; ++tq)
        for (int64_t c2 = 0; c2 < hd; ++c2) {
          const int64_t dst_row = s * 3 * hd + tq * hd + c2;
          const int64_t src_row = tq * D + (int64_t)ho[s] * hd + c2;
          for (int64_t j = 0; j < D; ++j)
            wr.mat(o(ELASTO_T_WQKV), dst_row * D + j, qkv_w[src_row * D + ev[j]]);
          wr.vec(o(ELASTO_T_BQKV), dst_row, qkv_b[src_row]);
        }
    const float* proj_w = w.proj_w + (int64_t)l * D * D;
    for (int64_t j = 0; j < D; ++j)
      for (int64_t s = 0; s < H; ++s)
        for (int64_t c2 = 0; c2 < hd; ++c2)
          wr.mat(o(ELASTO_T_WO), j * D + s * hd + c2, proj_w[ev[j] * D + (int64_t)ho[s] * hd + c2]);
    const float* fc1_w = w.fc1_w + (int64_t)l * M * D;
    const float* fc1_b = w.fc1_b + (int64_t)l * M;
    for (int64_t s = 0; s < M; ++s) {
      for (int64_t j = 0; j < D; ++j) wr.mat(o(ELASTO_T_W1), s * D + j, fc1_w[(int64_t)mo[s] * D + ev[j]]);
      wr.vec(o(ELASTO_T_B1), s, fc1_b[mo[s]]);
    }
    const float* fc2_w = w.fc2_w + (int64_t)l * D * M;
    for (int64_t j = 0; j < D; ++j)
      for (int64_t s = 0; s < M; ++s) wr.mat(o(ELASTO_T_W2), j * M + s, fc2_w[ev[j] * M + mo[s]]);
  }
}

double mode_flops(const elasto_config_t& c, const int32_t* nh, const int32_t* nm, int embed) {
  const Dims d = dims_of(c);
  const double T = d.T, E = embed, hd = d.hd, Np = (double)d.grid * d.grid;
  double f = 2.0 * Np * d.patch_k * E + 2.0 * E * c.num_classes;
  for (int l = 0; l < c.depth; ++l) {
    const double h = nh[l], m = nm[l];
    f += 2.0 * T * (4.0 * hd * h * E + 2.0 * E * m) + 2.0 * 2.0 * T * T * hd * h;
  }
  return f;
}

int64_t mode_weight_bytes(const elasto_config_t& c, const int32_t* nh, const int32_t* nm,
                          int embed) {
  const Dims d = dims_of(c);
  const int64_t me = c.dtype == ELASTO_BF16 ? 2 : 4, E = embed, hd = d.hd;
  int64_t e = E * d.patch_k + (int64_t)c.num_classes * E;
  for (int l = 0; l < c.depth; ++l) e += 4 * hd * nh[l] * E + 2 * E * (int64_t)nm[l];
  return e * me;
}

}  // namespace elasto

using namespace elasto;

extern "C" {

const char* elasto_last_error(void) { return g_err.c_str(); }

elasto_status_t elasto_validate(const elasto_config_t* cfg, const elasto_dn_table_t* table) {
  if (!cfg || !table) return fail(ELASTO_ERR_INVALID_ARG, "%s is NULL", cfg ? "DN table" : "config");
  if (!check_config(cfg)) return ELASTO_ERR_BAD_CONFIG;
  if (!check_table(cfg, table)) return ELASTO_ERR_BAD_TABLE;
  clear_error();
  return ELASTO_OK;
}

elasto_status_t elasto_packed_bytes(const elasto_config_t* cfg, int64_t* bytes) {
  if (!bytes) return fail(ELASTO_ERR_INVALID_ARG, "bytes is NULL");
  if (!check_config(cfg)) return ELASTO_ERR_BAD_CONFIG;
  *bytes = make_layout(*cfg).total;
  return ELASTO_OK;
}

elasto_status_t elasto_packed_layout(const elasto_config_t* cfg, int32_t tensor, int32_t layer,
                                     int64_t* offset, int64_t* rows, int64_t* cols,
                                     int32_t* elem_bytes) {
  if (!offset || !rows || !cols || !elem_bytes) return fail(ELASTO_ERR_INVALID_ARG, "NULL output pointer");
  if (!check_config(cfg)) return ELASTO_ERR_BAD_CONFIG;
  if (tensor < 0 || tensor >= ELASTO_T_COUNT) return fail(ELASTO_ERR_INVALID_ARG, "tensor id %d out of range", tensor);
  if (tensor >= ELASTO_T_LN1_G && (layer < 0 || layer >= cfg->depth))
    return fail(ELASTO_ERR_INVALID_ARG, "layer %d out of range", layer);
  const TensorSpec s = make_layout(*cfg).get(tensor, tensor >= ELASTO_T_LN1_G ? layer : 0);
  *offset = s.offset;
  *rows = s.rows;
  *cols = s.cols;
  *elem_bytes = s.elem_bytes;
  return ELASTO_OK;
}

elasto_status_t elasto_pack_weights(const elasto_config_t* cfg, const elasto_weights_t* w,
                                    const elasto_dn_table_t* table, void* dst, int64_t dst_bytes) {
  if (!check_config(cfg)) return ELASTO_ERR_BAD_CONFIG;
  if (!check_table(cfg, table)) return ELASTO_ERR_BAD_TABLE;
  if (!check_weights(w)) return ELASTO_ERR_INVALID_ARG;
  if (!dst) return fail(ELASTO_ERR_INVALID_ARG, "dst is NULL");
  const Layout L = make_layout(*cfg);
  if (dst_bytes < L.total) return fail(ELASTO_ERR_INVALID_ARG, "dst_bytes %lld < %lld", (long long)dst_bytes, (long long)L.total);
  pack(*cfg, *w, *table, L, static_cast<uint8_t*>(dst));
  clear_error();
  return ELASTO_OK;
}

}  // extern "C"
