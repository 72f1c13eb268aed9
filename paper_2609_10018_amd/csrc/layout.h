// Host-only part of the library: config / DN-table validation, the packed
// prefix layout of the weights, packing (with fp32 -> bf16 rounding) and the
// thread-local error message.  No HIP call is made here, so this unit builds
// and runs without a GPU (and under host sanitizers).
#pragma once

#include <stdint.h>

#include <string>

#include "../../include/elasto.h"

namespace elasto {

struct TensorSpec {
  int64_t offset;  // bytes from the start of the packed image
  int64_t rows, cols;
  int32_t elem_bytes;
};

struct Layout {
  TensorSpec global[ELASTO_T_LN1_G];                       // ids below ELASTO_T_LN1_G
  int64_t layer_base = 0, layer_stride = 0;                // bytes
  TensorSpec layer[ELASTO_T_COUNT - ELASTO_T_LN1_G];       // offsets relative to the layer
  int64_t total = 0;
  TensorSpec get(int tensor, int layer_idx) const;
};

struct Dims {
  int T, hd, grid, patch_k;
};

Dims dims_of(const elasto_config_t& c);

// Return false and set the thread-local error on failure.
bool check_config(const elasto_config_t* cfg);
bool check_table(const elasto_config_t* cfg, const elasto_dn_table_t* t);
Layout make_layout(const elasto_config_t& cfg);
void pack(const elasto_config_t& cfg, const elasto_weights_t& w, const elasto_dn_table_t& t,
          const Layout& lay, uint8_t* dst);
bool check_weights(const elasto_weights_t* w);

uint16_t f32_to_bf16_rne(float f);

void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();
elasto_status_t fail(elasto_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Per-image FLOPs of a mode (2 x MACs of every contraction) with per-layer
// head / unit counts and embed active embedding channels.
double mode_flops(const elasto_config_t& cfg, const int32_t* n_heads_k, const int32_t* n_mlp_k,
                  int embed);
// Bytes of the weight matrices the mode reads.
int64_t mode_weight_bytes(const elasto_config_t& cfg, const int32_t* n_heads_k,
                          const int32_t* n_mlp_k, int embed);

}  // namespace elasto
