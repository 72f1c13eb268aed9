// Internal: the ViT handle behind elasto_handle_t, shared by the forward
// (api.cpp) and the growth step (growth.cpp).
#pragma once

#include <hip/hip_runtime.h>

#include <vector>

#include "layout.h"

struct elasto_handle_s {
  using Dims = elasto::Dims;
  using Layout = elasto::Layout;
  elasto_config_t cfg;
  Dims dims;
  Layout lay;
  int device = 0;
  int num_modes = 0;
  std::vector<int32_t> n_heads, n_mlp;  // [num_modes][depth]
  std::vector<int32_t> n_embed;         // [num_modes] active embedding channels
  int mode = 0;
  uint8_t* dw = nullptr;  // packed weights
  uint8_t* ds = nullptr;  // activation scratch
  int64_t wbytes = 0, sbytes = 0;
  void *x = nullptr, *u = nullptr, *qkv = nullptr, *o = nullptr, *g = nullptr, *ucls = nullptr;
  float* xcls = nullptr;  // fp32 class-token rows of the residual stream (bf16 path)
  // kernel timing
  int timed_class = -1;
  std::vector<hipEvent_t> events;
  int used = 0;
  int64_t skipped = 0;
};

