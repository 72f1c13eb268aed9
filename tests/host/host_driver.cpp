// Drives the library's C ABI through the host sources only, linked against
// the counting HIP stand-ins of hip_stub.cpp.  Built with g++ and
// -fsanitize=address,undefined by tests/test_host_sanitized.py, so every
// validation path, the weight packing, the handle lifecycle (including
// allocation failures at each hipMalloc), the forward's host-side planning
// and the DN selection run under the host sanitizers.  It also checks that
// selecting a DN mode (elasto_set_mode, elasto_cnn_set_mode) makes no HIP
// call and launches nothing, and that a forward allocates nothing.
//
// Prints one line per failed check and ends with "host driver: N checks,
// F failed"; the exit status is 1 when any check failed.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <random>
#include <vector>

#include "../../include/elasto.h"
#include "hip_stub.h"

namespace {

int g_checks = 0, g_failed = 0;

void check(bool ok, const char* what, int line) {
  ++g_checks;
  if (!ok) {
    ++g_failed;
    printf("FAILED (line %d): %s -- last error: %s\n", line, what, elasto_last_error());
  }
}
#define CHECK(cond) check((cond), #cond, __LINE__)

std::mt19937 g_rng(1234);

std::vector<float> randn(size_t n, float std) {
  std::normal_distribution<float> d(0.f, std);
  std::vector<float> v(n);
  for (auto& x : v) x = d(g_rng);
  return v;
}

std::vector<int32_t> perm(int n, bool reversed) {
  std::vector<int32_t> p(n);
  for (int i = 0; i < n; ++i) p[i] = reversed ? n - 1 - i : i;
  return p;
}

// Host weights of a ViT config, canonical order (elasto_weights_t).
struct VitWeights {
  std::vector<float> patch_w, patch_b, cls, pos, ln1_g, ln1_b, qkv_w, qkv_b, proj_w, proj_b,
      ln2_g, ln2_b, fc1_w, fc1_b, fc2_w, fc2_b, norm_g, norm_b, head_w, head_b;
  elasto_weights_t w{};

  explicit VitWeights(const elasto_config_t& c) {
    const size_t d = c.dim, L = c.depth, M = c.mlp_hidden, C = c.num_classes, P = c.patch;
    const size_t T = (size_t)(c.img / c.patch) * (c.img / c.patch) + 1;
    patch_w = randn(d * c.in_chans * P * P, 0.02f);
    patch_b = randn(d, 0.02f);
    cls = randn(d, 0.02f);
    pos = randn(T * d, 0.02f);
    ln1_g = randn(L * d, 0.1f);
    ln1_b = randn(L * d, 0.1f);
    qkv_w = randn(L * 3 * d * d, 0.02f);
    qkv_b = randn(L * 3 * d, 0.02f);
    proj_w = randn(L * d * d, 0.02f);
    proj_b = randn(L * d, 0.02f);
    ln2_g = randn(L * d, 0.1f);
    ln2_b = randn(L * d, 0.1f);
    fc1_w = randn(L * M * d, 0.02f);
    fc1_b = randn(L * M, 0.02f);
    fc2_w = randn(L * d * M, 0.02f);
    fc2_b = randn(L * d, 0.02f);
    norm_g = randn(d, 0.1f);
    norm_b = randn(d, 0.1f);
    head_w = randn(C * d, 0.02f);
    head_b = randn(C, 0.02f);
    w = {patch_w.data(), patch_b.data(), cls.data(), pos.data(), ln1_g.data(), ln1_b.data(),
         qkv_w.data(), qkv_b.data(), proj_w.data(), proj_b.data(), ln2_g.data(), ln2_b.data(),
         fc1_w.data(), fc1_b.data(), fc2_w.data(), fc2_b.data(), norm_g.data(), norm_b.data(),
         head_w.data(), head_b.data()};
  }
};

// Nested DN table: mode k keeps max(1, heads >> k) heads and mlp >> k units
// (and, with embed, dim >> k channels rounded to 8).
struct VitTable {
  std::vector<int32_t> n_heads, n_mlp, head_order, mlp_order, n_embed, embed_order;
  elasto_dn_table_t t{};

  VitTable(const elasto_config_t& c, int modes, bool embed) {
    for (int k = 0; k < modes; ++k)
      for (int l = 0; l < c.depth; ++l) {
        n_heads.push_back(c.heads >> k > 0 ? c.heads >> k : 1);
        n_mlp.push_back(c.mlp_hidden >> k > 0 ? c.mlp_hidden >> k : 1);
      }
    for (int l = 0; l < c.depth; ++l) {
      auto h = perm(c.heads, l % 2), m = perm(c.mlp_hidden, l % 2 == 0);
      head_order.insert(head_order.end(), h.begin(), h.end());
      mlp_order.insert(mlp_order.end(), m.begin(), m.end());
    }
    if (embed) {
      for (int k = 0; k < modes; ++k) n_embed.push_back(((c.dim >> k) + 7) / 8 * 8);
      embed_order = perm(c.dim, true);
    }
    t = {modes, c.depth, n_heads.data(), n_mlp.data(), head_order.data(), mlp_order.data(),
         embed ? n_embed.data() : nullptr, embed ? embed_order.data() : nullptr};
  }
};

elasto_config_t vit_config(int32_t dtype) {
  elasto_config_t c{};
  c.img = 32;
  c.patch = 8;
  c.in_chans = 3;
  c.dim = dtype == ELASTO_BF16 ? 128 : 64;  // bf16 needs head_dim 64
  c.depth = 2;
  c.heads = 2;
  c.mlp_hidden = dtype == ELASTO_BF16 ? 256 : 128;
  c.num_classes = 10;
  c.max_batch = 4;
  c.dtype = dtype;
  c.ln_eps = 1e-6f;
  return c;
}

void test_validation(int32_t dtype) {
  elasto_config_t c = vit_config(dtype);
  VitTable tab(c, 3, dtype == ELASTO_BF16);
  hipstub_reset_counts();
  CHECK(elasto_validate(&c, &tab.t) == ELASTO_OK);

  {  // bad tables
    VitTable t(c, 3, dtype == ELASTO_BF16);
    t.n_heads[1] = 0;
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
  }
  {
    VitTable t(c, 3, dtype == ELASTO_BF16);
    t.n_mlp[2] = c.mlp_hidden + 1;
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
  }
  {
    VitTable t(c, 3, dtype == ELASTO_BF16);
    t.mlp_order[5] = t.mlp_order[6];
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
  }
  {
    VitTable t(c, 3, dtype == ELASTO_BF16);
    t.head_order[0] = -1;
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
  }
  {
    VitTable t(c, 3, dtype == ELASTO_BF16);
    t.t.depth = c.depth + 1;
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
  }
  {
    VitTable t(c, 3, true);
    t.n_embed[1] = c.dim + 8;
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
    t.n_embed[1] = 0;
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
  }
  {
    VitTable t(c, 3, false);
    t.t.num_modes = 0;
    CHECK(elasto_validate(&c, &t.t) == ELASTO_ERR_BAD_TABLE);
  }
  // bad configs
  int32_t elasto_config_t::*const fields[] = {&elasto_config_t::img, &elasto_config_t::dim,
                                        &elasto_config_t::mlp_hidden,
                                        &elasto_config_t::depth, &elasto_config_t::heads};
  for (auto f : fields) {
    elasto_config_t b = c;
    b.*f = 0;
    CHECK(elasto_validate(&b, &tab.t) != ELASTO_OK);
    b.*f = -5;
    CHECK(elasto_validate(&b, &tab.t) != ELASTO_OK);
  }
  {
    elasto_config_t b = c;
    b.img = 30;  // not a multiple of the patch
    CHECK(elasto_validate(&b, &tab.t) == ELASTO_ERR_BAD_CONFIG);
    b = c;
    b.ln_eps = 0.f;
    CHECK(elasto_validate(&b, &tab.t) == ELASTO_ERR_BAD_CONFIG);
    b = c;
    b.ln_eps = NAN;
    CHECK(elasto_validate(&b, &tab.t) == ELASTO_ERR_BAD_CONFIG);
    b = c;
    b.dtype = 7;
    CHECK(elasto_validate(&b, &tab.t) == ELASTO_ERR_BAD_CONFIG);
    b = c;
    b.dim = 4096;
    CHECK(elasto_validate(&b, &tab.t) != ELASTO_OK);
  }
  CHECK(elasto_validate(nullptr, &tab.t) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_validate(&c, nullptr) == ELASTO_ERR_INVALID_ARG);
  CHECK(hipstub_api_calls() == 0 && hipstub_launches() == 0);
}

void test_packing(int32_t dtype) {
  elasto_config_t c = vit_config(dtype);
  VitWeights w(c);
  VitTable tab(c, 3, true);
  int64_t bytes = 0;
  CHECK(elasto_packed_bytes(&c, &bytes) == ELASTO_OK && bytes > 0);
  std::vector<uint8_t> buf(bytes);
  CHECK(elasto_pack_weights(&c, &w.w, &tab.t, buf.data(), bytes - 1) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_pack_weights(&c, &w.w, &tab.t, buf.data(), bytes) == ELASTO_OK);
  for (int t = 0; t < ELASTO_T_COUNT; ++t)
    for (int l = 0; l < c.depth; ++l) {
      int64_t off, rows, cols;
      int32_t eb;
      CHECK(elasto_packed_layout(&c, t, l, &off, &rows, &cols, &eb) == ELASTO_OK);
      CHECK(off >= 0 && off + rows * cols * eb <= bytes && off % 256 == 0);
    }
  int64_t off, rows, cols;
  int32_t eb;
  CHECK(elasto_packed_layout(&c, ELASTO_T_COUNT, 0, &off, &rows, &cols, &eb) != ELASTO_OK);
  CHECK(elasto_packed_layout(&c, ELASTO_T_WQKV, c.depth, &off, &rows, &cols, &eb) != ELASTO_OK);
  elasto_weights_t nw = w.w;
  nw.fc2_w = nullptr;
  CHECK(elasto_pack_weights(&c, &nw, &tab.t, buf.data(), bytes) == ELASTO_ERR_INVALID_ARG);
}

// Creates a handle, checks mode switching makes no HIP call, runs forwards
// through every entry point and destroys it.
void test_lifecycle(int32_t dtype, bool embed) {
  elasto_config_t c = vit_config(dtype);
  VitWeights w(c);
  VitTable tab(c, 3, embed);
  const long live0 = hipstub_live_allocations();

  hipstub_reset_counts();
  elasto_handle_t h = nullptr;
  CHECK(elasto_create(nullptr, &w.w, &tab.t, &h) == ELASTO_ERR_INVALID_ARG && !h);
  CHECK(elasto_create(&c, nullptr, &tab.t, &h) == ELASTO_ERR_INVALID_ARG && !h);
  CHECK(elasto_create(&c, &w.w, nullptr, &h) == ELASTO_ERR_INVALID_ARG && !h);
  CHECK(elasto_create(&c, &w.w, &tab.t, nullptr) == ELASTO_ERR_INVALID_ARG);
  CHECK(hipstub_api_calls() == 0);
  CHECK(elasto_create(&c, &w.w, &tab.t, &h) == ELASTO_OK && h);
  if (!h) return;
  const long create_mallocs = hipstub_mallocs();
  CHECK(create_mallocs >= 2);

  // Mode switching: an O(1) host store.
  hipstub_reset_counts();
  for (int rep = 0; rep < 1000; ++rep)
    for (int k = 0; k < 3; ++k) {
      CHECK(elasto_set_mode(h, k) == ELASTO_OK);
      int32_t got = -1;
      CHECK(elasto_get_mode(h, &got) == ELASTO_OK && got == k);
    }
  CHECK(elasto_set_mode(h, 3) == ELASTO_ERR_MODE_RANGE);
  CHECK(elasto_set_mode(h, -1) == ELASTO_ERR_MODE_RANGE);
  CHECK(hipstub_api_calls() == 0);
  CHECK(hipstub_launches() == 0);

  // Forwards: every mode and batch, no allocation.
  const size_t T = (size_t)(c.img / c.patch) * (c.img / c.patch) + 1;
  (void)T;
  const size_t img_elems = (size_t)c.max_batch * c.in_chans * c.img * c.img;
  std::vector<uint8_t> images(img_elems * 4, 0);
  std::vector<float> logits((size_t)c.max_batch * c.num_classes);
  hipstub_reset_counts();
  CHECK(elasto_forward(h, images.data(), 0, logits.data(), nullptr) == ELASTO_ERR_BATCH_RANGE);
  CHECK(elasto_forward(h, images.data(), c.max_batch + 1, logits.data(), nullptr) ==
        ELASTO_ERR_BATCH_RANGE);
  CHECK(elasto_forward(h, nullptr, 1, logits.data(), nullptr) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_forward(h, images.data(), 1, nullptr, nullptr) == ELASTO_ERR_INVALID_ARG);
  CHECK(hipstub_launches() == 0);
  for (int k = 0; k < 3; ++k)
    for (int b = 1; b <= c.max_batch; ++b) {
      CHECK(elasto_set_mode(h, k) == ELASTO_OK);
      hipstub_reset_counts();
      CHECK(elasto_forward(h, images.data(), b, logits.data(), nullptr) == ELASTO_OK);
      CHECK(hipstub_launches() > 0 && hipstub_mallocs() == 0);
      if (dtype == ELASTO_BF16) {
        hipstub_reset_counts();
        CHECK(elasto_forward_static(h, images.data(), b, logits.data(), nullptr) == ELASTO_OK);
        CHECK(hipstub_launches() > 0 && hipstub_mallocs() == 0);
      }
    }
  CHECK(elasto_forward_static(h, images.data(), c.max_batch + 1, logits.data(), nullptr) ==
        ELASTO_ERR_BATCH_RANGE);

  // Cost queries.
  for (int k = 0; k < 3; ++k) {
    double flops = 0;
    int64_t wb = 0;
    CHECK(elasto_mode_info(h, k, &flops, &wb) == ELASTO_OK && flops > 0 && wb > 0);
    for (int kc = 0; kc < ELASTO_K_COUNT; ++kc) {
      double f = -1, b = -1;
      int32_t n = -1;
      CHECK(elasto_kernel_work(h, k, 2, kc, &f, &b, &n) == ELASTO_OK && f >= 0 && b >= 0 &&
            n >= 1);
    }
  }
  double f;
  int64_t wb, sb;
  CHECK(elasto_mode_info(h, 3, &f, &wb) == ELASTO_ERR_MODE_RANGE);
  CHECK(elasto_memory_info(h, &wb, &sb) == ELASTO_OK && wb > 0 && sb > 0);

  // Per-kernel timing and mode profiling (events only).
  CHECK(elasto_kernel_timing(h, ELASTO_K_FC1, 8) == ELASTO_OK);
  CHECK(elasto_forward(h, images.data(), 2, logits.data(), nullptr) == ELASTO_OK);
  double ms = 0;
  int64_t launches = 0;
  CHECK(elasto_kernel_timing_read(h, &ms, &launches) == ELASTO_OK && launches == c.depth);
  CHECK(elasto_kernel_timing(h, -1, 0) == ELASTO_OK);
  CHECK(elasto_kernel_timing(h, ELASTO_K_COUNT, 8) == ELASTO_ERR_INVALID_ARG);
  std::vector<double> lat(3), mem(3), fl(3);
  CHECK(elasto_set_mode(h, 1) == ELASTO_OK);
  CHECK(elasto_profile_modes(h, images.data(), 2, logits.data(), 1, 3, nullptr, lat.data(),
                             mem.data(), fl.data()) == ELASTO_OK);
  int32_t mode = -1;
  CHECK(elasto_get_mode(h, &mode) == ELASTO_OK && mode == 1);
  CHECK(fl[0] > fl[1] && fl[1] > fl[2] && mem[0] > mem[2]);
  CHECK(elasto_profile_modes(h, images.data(), 2, logits.data(), 1, 0, nullptr, lat.data(),
                             mem.data(), fl.data()) == ELASTO_ERR_INVALID_ARG);

  hipstub_reset_counts();
  CHECK(elasto_destroy(h) == ELASTO_OK);
  CHECK(hipstub_live_allocations() == live0);

  // Allocation failure at every hipMalloc of create: an error, no handle,
  // nothing left allocated.
  for (long i = 0; i < create_mallocs; ++i) {
    hipstub_fail_malloc_at(i);
    elasto_handle_t h2 = nullptr;
    CHECK(elasto_create(&c, &w.w, &tab.t, &h2) == ELASTO_ERR_OUT_OF_MEMORY);
    CHECK(h2 == nullptr);
    CHECK(hipstub_live_allocations() == live0);
  }
  hipstub_fail_malloc_at(-1);
}

void test_growth() {
  elasto_config_t c = vit_config(ELASTO_BF16);
  VitWeights w(c);
  VitTable tab(c, 3, false);
  elasto_handle_t h = nullptr;
  CHECK(elasto_create(&c, &w.w, &tab.t, &h) == ELASTO_OK);
  if (!h) return;
  const long live0 = hipstub_live_allocations();
  hipstub_reset_counts();
  elasto_growth_t g = nullptr;
  CHECK(elasto_growth_create(h, 0, &g) == ELASTO_ERR_BATCH_RANGE || g == nullptr);
  CHECK(elasto_growth_create(h, 2, &g) == ELASTO_OK && g);
  const long mallocs = hipstub_mallocs();
  std::vector<uint8_t> images((size_t)2 * c.in_chans * c.img * c.img * 2, 0);
  std::vector<int32_t> labels = {1, 2};
  std::vector<float> stats(3);
  if (g) {
    CHECK(elasto_growth_step(g, 0, images.data(), labels.data(), 2, 1e-3f, 1.f, stats.data(),
                             nullptr) == ELASTO_OK);
    CHECK(elasto_growth_step(g, 2, images.data(), labels.data(), 2, 1e-3f, 1.f, stats.data(),
                             nullptr) != ELASTO_OK);  // last mode has no smaller one
    CHECK(elasto_growth_step(g, 0, images.data(), labels.data(), 3, 1e-3f, 1.f, stats.data(),
                             nullptr) == ELASTO_ERR_BATCH_RANGE);
    CHECK(elasto_growth_step(g, 0, images.data(), labels.data(), 2, NAN, 1.f, stats.data(),
                             nullptr) == ELASTO_ERR_INVALID_ARG);
    CHECK(elasto_growth_step(g, 0, images.data(), labels.data(), 2, 1e-3f, 0.f, stats.data(),
                             nullptr) == ELASTO_ERR_INVALID_ARG);
    int64_t bytes = 0;
    CHECK(elasto_packed_bytes(&c, &bytes) == ELASTO_OK);
    std::vector<uint8_t> packed(bytes);
    std::vector<float> masters(bytes / 2);
    CHECK(elasto_growth_read(g, 0, packed.data(), bytes) == ELASTO_OK);
    CHECK(elasto_growth_read(g, 1, masters.data(), bytes * 2) == ELASTO_OK);
    CHECK(elasto_growth_read(g, 0, packed.data(), bytes - 2) == ELASTO_ERR_INVALID_ARG);
    CHECK(elasto_growth_read(g, 2, packed.data(), bytes) == ELASTO_ERR_INVALID_ARG);
    CHECK(elasto_growth_destroy(g) == ELASTO_OK);
  }
  CHECK(hipstub_live_allocations() == live0);
  for (long i = 0; i < mallocs; ++i) {
    hipstub_fail_malloc_at(i);
    elasto_growth_t g2 = nullptr;
    CHECK(elasto_growth_create(h, 2, &g2) == ELASTO_ERR_OUT_OF_MEMORY && g2 == nullptr);
    CHECK(hipstub_live_allocations() == live0);
  }
  hipstub_fail_malloc_at(-1);
  CHECK(elasto_destroy(h) == ELASTO_OK);

  // The growth step needs a bf16 handle.
  elasto_config_t cf = vit_config(ELASTO_FP32);
  VitWeights wf(cf);
  VitTable tf(cf, 2, false);
  elasto_handle_t hf = nullptr;
  CHECK(elasto_create(&cf, &wf.w, &tf.t, &hf) == ELASTO_OK);
  elasto_growth_t gf = nullptr;
  CHECK(elasto_growth_create(hf, 2, &gf) == ELASTO_ERR_BAD_CONFIG && gf == nullptr);
  CHECK(elasto_destroy(hf) == ELASTO_OK);
}

void test_ops() {
  std::vector<uint8_t> a(1 << 16), b(1 << 16), o(1 << 16);
  std::vector<float> g(256, 1.f), bias(256, 0.f);
  hipstub_reset_counts();
  // LayerNorm: bad dtype, rows, d, eps.
  CHECK(elasto_op_layernorm(5, a.data(), 64, nullptr, 1, o.data(), 4, 64, g.data(), bias.data(),
                            1e-6f, nullptr) != ELASTO_OK);
  CHECK(elasto_op_layernorm(ELASTO_BF16, a.data(), 64, nullptr, 1, o.data(), 4, 60, g.data(),
                            bias.data(), 1e-6f, nullptr) != ELASTO_OK);
  CHECK(elasto_op_layernorm(ELASTO_FP32, a.data(), 64, g.data(), 1, o.data(), 4, 64, g.data(),
                            bias.data(), 1e-6f, nullptr) != ELASTO_OK);
  // Linear: bad epilogue, a row stride that breaks 16-byte rows, null operand.
  CHECK(elasto_op_linear(ELASTO_BF16, 9, a.data(), 64, b.data(), 64, o.data(), 64, nullptr, 1,
                         bias.data(), 4, 64, 64, nullptr) != ELASTO_OK);
  CHECK(elasto_op_linear(ELASTO_BF16, ELASTO_EPI_BIAS, a.data(), 60, b.data(), 64, o.data(), 64,
                         nullptr, 1, bias.data(), 4, 64, 60, nullptr) != ELASTO_OK);
  CHECK(elasto_op_linear(ELASTO_BF16, ELASTO_EPI_BIAS, nullptr, 64, b.data(), 64, o.data(), 64,
                         nullptr, 1, bias.data(), 4, 64, 64, nullptr) != ELASTO_OK);
  // Attention: head_dim other than 64 on the bf16 path.
  CHECK(elasto_op_attention(ELASTO_BF16, a.data(), 3 * 2 * 32, o.data(), 64, 1, 5, 2, 32, 0.1f,
                            nullptr) != ELASTO_OK);
  // Convolution: channels not a multiple of 8.
  CHECK(elasto_op_conv2d(a.data(), 1, 4, 4, 12, 12, 3, 3, 1, 1, b.data(), 9 * 16, 16,
                         bias.data(), o.data(), 16, 16, 1, nullptr) != ELASTO_OK);
  CHECK(hipstub_api_calls() == 0 && hipstub_launches() == 0);

  // Valid calls launch.
  CHECK(elasto_op_layernorm(ELASTO_BF16, a.data(), 64, nullptr, 1, o.data(), 4, 64, g.data(),
                            bias.data(), 1e-6f, nullptr) == ELASTO_OK);
  CHECK(elasto_op_linear(ELASTO_BF16, ELASTO_EPI_BIAS_GELU, a.data(), 64, b.data(), 64, o.data(),
                         64, nullptr, 1, bias.data(), 4, 64, 64, nullptr) == ELASTO_OK);
  CHECK(elasto_op_linear(ELASTO_FP32, ELASTO_EPI_BIAS, a.data(), 64, b.data(), 64, o.data(), 64,
                         nullptr, 1, bias.data(), 4, 64, 64, nullptr) == ELASTO_OK);
  // Ragged K (a K-sliced weight of a narrow mode) is accepted on the bf16 path.
  CHECK(elasto_op_linear(ELASTO_BF16, ELASTO_EPI_BIAS, a.data(), 64, b.data(), 64, o.data(), 64,
                         nullptr, 1, bias.data(), 4, 64, 60, nullptr) == ELASTO_OK);
  CHECK(elasto_op_attention(ELASTO_BF16, a.data(), 3 * 2 * 64, o.data(), 128, 1, 5, 2, 64, 0.125f,
                            nullptr) == ELASTO_OK);
  CHECK(elasto_op_conv2d(a.data(), 1, 4, 4, 16, 16, 3, 3, 1, 1, b.data(), 9 * 16, 16, bias.data(),
                         o.data(), 16, 16, 1, nullptr) == ELASTO_OK);
  CHECK(hipstub_launches() >= 5);
}

void test_select() {
  // Eq. 11 against a brute-force scan on random tables.
  std::uniform_real_distribution<double> u(0.0, 1.0);
  for (int rep = 0; rep < 200; ++rep) {
    const int n = 1 + rep % 7;
    std::vector<double> fl(n), lat(n), mem(n), acc(n), pw(n);
    for (int k = 0; k < n; ++k) {
      fl[k] = floor(u(g_rng) * 5);  // ties
      lat[k] = u(g_rng);
      mem[k] = u(g_rng);
      acc[k] = u(g_rng);
      pw[k] = u(g_rng);
    }
    elasto_dn_lut_t lut{n, fl.data(), lat.data(), mem.data(), acc.data(), pw.data()};
    const double bl = u(g_rng), bm = u(g_rng), ba = u(g_rng) * 0.5, bp = u(g_rng);
    int best = -1;
    for (int k = 0; k < n; ++k)
      if (lat[k] <= bl && mem[k] <= bm && acc[k] >= ba && pw[k] <= bp &&
          (best < 0 || fl[k] < fl[best]))
        best = k;
    int32_t got = -2;
    const elasto_status_t st = elasto_select_mode(&lut, bl, bm, ba, bp, &got);
    CHECK(got == best);
    CHECK(st == (best < 0 ? ELASTO_ERR_INFEASIBLE : ELASTO_OK));
  }
  double v[2] = {1, 2}, bad[2] = {1, NAN};
  elasto_dn_lut_t lut{2, v, v, v, nullptr, nullptr};
  int32_t m;
  CHECK(elasto_select_mode(&lut, INFINITY, INFINITY, -INFINITY, INFINITY, &m) == ELASTO_OK &&
        m == 0);
  CHECK(elasto_select_mode(&lut, INFINITY, INFINITY, 0.5, INFINITY, &m) ==
        ELASTO_ERR_INVALID_ARG);  // an accuracy bound with no accuracy column
  CHECK(elasto_select_mode(&lut, NAN, INFINITY, -INFINITY, INFINITY, &m) ==
        ELASTO_ERR_INVALID_ARG);
  elasto_dn_lut_t nan_lut{2, v, bad, v, nullptr, nullptr};
  CHECK(elasto_select_mode(&nan_lut, INFINITY, INFINITY, -INFINITY, INFINITY, &m) ==
        ELASTO_ERR_INVALID_ARG);
  elasto_dn_lut_t empty{0, v, v, v, nullptr, nullptr};
  CHECK(elasto_select_mode(&empty, INFINITY, INFINITY, -INFINITY, INFINITY, &m) ==
        ELASTO_ERR_INVALID_ARG);
}

// Elastic bottleneck ResNet: two stages of one block each.
struct Cnn {
  elasto_cnn_config_t c{};
  std::vector<std::vector<float>> tensors;
  std::vector<const float*> ptrs;
  std::vector<int32_t> n_width, order1, order2;
  elasto_cnn_weights_t w{};
  elasto_cnn_table_t t{};

  Cnn() {
    c.img = 64;
    c.in_chans = 3;
    c.stem = 16;
    c.num_stages = 2;
    c.widths[0] = 16;
    c.widths[1] = 32;
    c.blocks[0] = c.blocks[1] = 1;
    c.expansion = 4;
    c.num_classes = 10;
    c.max_batch = 2;
    c.dtype = ELASTO_BF16;
    auto add = [&](size_t n) { tensors.push_back(randn(n, 0.05f)); };
    add((size_t)c.stem * c.in_chans * 49);
    add(c.stem);
    int c_in = c.stem;
    for (int s = 0; s < c.num_stages; ++s) {
      const int wd = c.widths[s], co = wd * c.expansion;
      add((size_t)wd * c_in);
      add(wd);
      add((size_t)wd * wd * 9);
      add(wd);
      add((size_t)co * wd);
      add(co);
      add((size_t)co * c_in);  // projection shortcut on each stage's first block
      add(co);
      c_in = co;
    }
    add((size_t)c.num_classes * c_in);
    add(c.num_classes);
    for (auto& v : tensors) ptrs.push_back(v.data());
    w = {(int32_t)ptrs.size(), ptrs.data()};
    n_width = {16, 32, 8, 16};
    for (int s = 0; s < c.num_stages; ++s) {
      auto p1 = perm(c.widths[s], true), p2 = perm(c.widths[s], false);
      order1.insert(order1.end(), p1.begin(), p1.end());
      order2.insert(order2.end(), p2.begin(), p2.end());
    }
    t = {2, 2, n_width.data(), order1.data(), order2.data()};
  }
};

void test_cnn() {
  Cnn n;
  hipstub_reset_counts();
  CHECK(elasto_cnn_validate(&n.c, &n.t) == ELASTO_OK);
  {
    Cnn b;
    b.n_width[2] = 12;  // not a multiple of 8
    CHECK(elasto_cnn_validate(&b.c, &b.t) == ELASTO_ERR_BAD_TABLE);
    b.n_width[2] = 0;
    CHECK(elasto_cnn_validate(&b.c, &b.t) == ELASTO_ERR_BAD_TABLE);
    b.n_width[2] = 8;
    b.order2[3] = b.order2[4];
    CHECK(elasto_cnn_validate(&b.c, &b.t) == ELASTO_ERR_BAD_TABLE);
  }
  {
    Cnn b;
    b.c.img = 48;  // not a multiple of 32
    CHECK(elasto_cnn_validate(&b.c, &b.t) == ELASTO_ERR_BAD_CONFIG);
    b.c.img = 64;
    b.c.num_stages = 9;
    CHECK(elasto_cnn_validate(&b.c, &b.t) == ELASTO_ERR_BAD_CONFIG);
  }
  {
    Cnn b;
    b.w.num_tensors -= 1;
    elasto_cnn_t h = nullptr;
    CHECK(elasto_cnn_create(&b.c, &b.w, &b.t, &h) != ELASTO_OK && h == nullptr);
  }
  CHECK(hipstub_api_calls() == 0);

  const long live0 = hipstub_live_allocations();
  hipstub_reset_counts();
  elasto_cnn_t h = nullptr;
  CHECK(elasto_cnn_validate(nullptr, &n.t) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_cnn_validate(&n.c, nullptr) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_cnn_create(nullptr, &n.w, &n.t, &h) == ELASTO_ERR_INVALID_ARG && !h);
  CHECK(elasto_cnn_create(&n.c, nullptr, &n.t, &h) == ELASTO_ERR_INVALID_ARG && !h);
  CHECK(elasto_cnn_create(&n.c, &n.w, nullptr, &h) == ELASTO_ERR_INVALID_ARG && !h);
  CHECK(hipstub_api_calls() == 0);
  CHECK(elasto_cnn_create(&n.c, &n.w, &n.t, &h) == ELASTO_OK && h);
  if (!h) return;
  const long mallocs = hipstub_mallocs();
  hipstub_reset_counts();
  for (int rep = 0; rep < 1000; ++rep)
    for (int k = 0; k < 2; ++k) {
      CHECK(elasto_cnn_set_mode(h, k) == ELASTO_OK);
      int32_t got = -1;
      CHECK(elasto_cnn_get_mode(h, &got) == ELASTO_OK && got == k);
    }
  CHECK(elasto_cnn_set_mode(h, 2) == ELASTO_ERR_MODE_RANGE);
  CHECK(hipstub_api_calls() == 0 && hipstub_launches() == 0);

  std::vector<uint8_t> images((size_t)2 * 3 * 64 * 64 * 2, 0);
  std::vector<float> logits(20);
  for (int k = 0; k < 2; ++k)
    for (int b = 1; b <= 2; ++b) {
      CHECK(elasto_cnn_set_mode(h, k) == ELASTO_OK);
      hipstub_reset_counts();
      CHECK(elasto_cnn_forward(h, images.data(), b, logits.data(), nullptr) == ELASTO_OK);
      CHECK(hipstub_launches() > 0 && hipstub_mallocs() == 0);
      double macs = 0;
      int64_t wb = 0;
      CHECK(elasto_cnn_mode_info(h, k, &macs, &wb) == ELASTO_OK && macs > 0 && wb > 0);
    }
  CHECK(elasto_cnn_forward(h, images.data(), 3, logits.data(), nullptr) ==
        ELASTO_ERR_BATCH_RANGE);
  CHECK(elasto_cnn_destroy(h) == ELASTO_OK);
  CHECK(hipstub_live_allocations() == live0);
  {
    // max_batch 32: create times every tile plan of every site (each timing
    // here smaller than the last, so plans other than the planner's are
    // kept); forwards of more than 16 images then use them.
    Cnn t;
    t.c.max_batch = 32;
    hipstub_elapsed_decreasing(1);
    hipstub_reset_counts();
    elasto_cnn_t ht = nullptr;
    CHECK(elasto_cnn_create(&t.c, &t.w, &t.t, &ht) == ELASTO_OK && ht);
    CHECK(hipstub_launches() > 2 * 7 * 9);  // two modes, seven plans, nine sites
    std::vector<uint8_t> im((size_t)32 * 3 * 64 * 64 * 2, 0);
    std::vector<float> lg((size_t)32 * 10);
    for (int b : {32, 16, 1}) {
      hipstub_reset_counts();
      CHECK(elasto_cnn_forward(ht, im.data(), b, lg.data(), nullptr) == ELASTO_OK);
      CHECK(hipstub_launches() > 0 && hipstub_mallocs() == 0);
    }
    CHECK(elasto_cnn_destroy(ht) == ELASTO_OK);
    CHECK(hipstub_live_allocations() == live0);
    hipstub_elapsed_decreasing(0);
  }
  for (long i = 0; i < mallocs; ++i) {
    hipstub_fail_malloc_at(i);
    elasto_cnn_t h2 = nullptr;
    CHECK(elasto_cnn_create(&n.c, &n.w, &n.t, &h2) == ELASTO_ERR_OUT_OF_MEMORY && h2 == nullptr);
    CHECK(hipstub_live_allocations() == live0);
  }
  hipstub_fail_malloc_at(-1);
}

void test_null_handles() {
  hipstub_reset_counts();
  CHECK(elasto_set_mode(nullptr, 0) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_forward(nullptr, nullptr, 1, nullptr, nullptr) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_forward_static(nullptr, nullptr, 1, nullptr, nullptr) == ELASTO_ERR_INVALID_ARG);
  CHECK(elasto_destroy(nullptr) == ELASTO_OK);
  CHECK(elasto_cnn_destroy(nullptr) == ELASTO_OK);
  CHECK(elasto_growth_destroy(nullptr) == ELASTO_OK);
  CHECK(elasto_cnn_set_mode(nullptr, 0) == ELASTO_ERR_INVALID_ARG);
  CHECK(hipstub_api_calls() == 0);
}

}  // namespace

// bf16 handles of max_batch >= 32 time every GEMM tile plan at create (each
// stand-in timing smaller than the last, so plans other than the planner's
// are kept); forwards of more than half of max_batch images use them.
void test_tuned_plans(bool embed) {
  elasto_config_t c = vit_config(ELASTO_BF16);
  c.max_batch = 32;
  VitWeights w(c);
  VitTable tab(c, 3, embed);
  const long live0 = hipstub_live_allocations();
  hipstub_elapsed_decreasing(1);
  hipstub_reset_counts();
  elasto_handle_t h = nullptr;
  CHECK(elasto_create(&c, &w.w, &tab.t, &h) == ELASTO_OK && h);
  if (!h) return;
  CHECK(hipstub_launches() > 7 * 6);  // at least every plan of the distinct GEMM shapes
  std::vector<uint8_t> images((size_t)c.max_batch * c.in_chans * c.img * c.img * 2, 0);
  std::vector<float> logits((size_t)c.max_batch * c.num_classes);
  for (int k = 0; k < 3; ++k)
    for (int b : {32, 16, 1}) {
      CHECK(elasto_set_mode(h, k) == ELASTO_OK);
      hipstub_reset_counts();
      CHECK(elasto_forward(h, images.data(), b, logits.data(), nullptr) == ELASTO_OK);
      CHECK(elasto_forward_static(h, images.data(), b, logits.data(), nullptr) == ELASTO_OK);
      CHECK(hipstub_launches() > 0 && hipstub_mallocs() == 0);
    }
  CHECK(elasto_destroy(h) == ELASTO_OK);
  CHECK(hipstub_live_allocations() == live0);
  hipstub_elapsed_decreasing(0);
}

int main() {
  test_validation(ELASTO_FP32);
  test_validation(ELASTO_BF16);
  test_packing(ELASTO_FP32);
  test_packing(ELASTO_BF16);
  test_lifecycle(ELASTO_FP32, false);
  test_lifecycle(ELASTO_FP32, true);
  test_lifecycle(ELASTO_BF16, false);
  test_lifecycle(ELASTO_BF16, true);
  test_tuned_plans(false);
  test_tuned_plans(true);
  test_growth();
  test_ops();
  test_select();
  test_cnn();
  test_null_handles();
  CHECK(hipstub_live_allocations() == 0);
  hipstub_release_static();
  printf("host driver: %d checks, %d failed\n", g_checks, g_failed);
  return g_failed ? 1 : 0;
}
