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
  // LayerNorms folded into the q/k/v and fc1 GEMMs (bf16 path).  Per layer:
  // gamma1 (x) WQKV [3d][d] and gamma2 (x) W1 [M][d] (bf16), then for each
  // distinct embedding width w: column sums and folded biases of both
  // ([nw][3d] + [nw][3d] + [nw][M] + [nw][M] fp32).
  uint8_t* dfold = nullptr;
  int64_t fold_bytes = 0, fold_stride = 0;
  int64_t fold_wq = 0, fold_w1 = 0, fold_sq = 0, fold_cq = 0, fold_s1 = 0, fold_c1 = 0;
  std::vector<int32_t> widths;     // distinct active embedding widths
  std::vector<int32_t> width_idx;  // [num_modes] index into widths
  float2* lnpart = nullptr;        // [max_batch * T][lnseg] per-segment LayerNorm statistics
  float* ws = nullptr;             // split-K workspace of small-batch GEMMs (bf16 path)
  int64_t ws_bytes = 0;
  int lnseg = 0;                   // 64-column segments of d, rounded up to even
  // bf16: tile plan per (mode, GEMM site), sites in forward order: patch
  // embedding, per layer q/k/v, projection, fc1, fc2, then the head; chosen
  // at create by timing (plans.h).  Empty: the planner everywhere.
  int nsites = 0;
  std::vector<uint8_t> plans, plans_half;  // whole forwards / half-batch parts
  // Per mode: run a forward of more than max_batch / 2 images as two halves,
  // the second on the side stream (chosen at create by timing).
  std::vector<uint8_t> split;
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  // kernel timing
  int timed_class = -1;
  std::vector<hipEvent_t> events;
  int used = 0;
  int64_t skipped = 0;
};

// Recompute the folded LayerNorm weights from the packed weights (after
// create, and after anything that changes the packed weights).
hipError_t refold(elasto_handle_s* h, hipStream_t s);
