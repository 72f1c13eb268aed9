// Host stand-ins for the HIP runtime calls and kernel launchers that the
// library's host sources (api.cpp, cnn.cpp, growth.cpp, layout.cpp,
// select.cpp) make, so those sources can be built with g++ and the host
// sanitizers and run without a GPU.
//
// "Device" memory is ordinary heap memory filled with a byte pattern; every
// runtime call and every launch is counted, hipMalloc can be made to fail at
// a chosen call, and outstanding allocations are tracked so a test can check
// that an error path or a destroy released everything it took.  Launchers
// only count: no kernel runs.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <map>

#include "hip_stub.h"
#include "../../paper_2609_10018_amd/csrc/kernels.h"

namespace {
long g_api_calls = 0;
long g_launches = 0;
long g_mallocs = 0;
long g_fail_at = -1;  // hipMalloc call index (0-based, counted from arming) that fails
long g_armed_mallocs = 0;
std::map<void*, size_t> g_live;
uint8_t* g_static = nullptr;
int g_elapsed_decreasing = 0;
float g_elapsed = 1000.0f;

void tick() { ++g_api_calls; }
hipError_t api() {
  tick();
  return hipSuccess;
}
hipError_t launch() {
  ++g_launches;
  return hipSuccess;
}
}  // namespace

extern "C" {
long hipstub_api_calls(void) { return g_api_calls; }
long hipstub_launches(void) { return g_launches; }
long hipstub_mallocs(void) { return g_mallocs; }
long hipstub_live_allocations(void) { return (long)g_live.size(); }
void hipstub_reset_counts(void) { g_api_calls = g_launches = g_mallocs = 0; }
void hipstub_elapsed_decreasing(int on) {
  g_elapsed_decreasing = on;
  g_elapsed = 1000.0f;
}
void hipstub_fail_malloc_at(long n) {
  g_fail_at = n;
  g_armed_mallocs = 0;
}
}

hipError_t hipMalloc(void** p, size_t n) {
  tick();
  ++g_mallocs;
  if (g_fail_at >= 0 && g_armed_mallocs++ == g_fail_at) {
    g_fail_at = -1;
    return hipErrorOutOfMemory;
  }
  void* q = malloc(n ? n : 1);
  if (!q) return hipErrorOutOfMemory;
  memset(q, 0xA5, n);
  g_live[q] = n;
  *p = q;
  return hipSuccess;
}

hipError_t hipFree(void* p) {
  tick();
  if (!p) return hipSuccess;
  auto it = g_live.find(p);
  if (it == g_live.end()) abort();  // freeing what hipMalloc never returned
  g_live.erase(it);
  free(p);
  return hipSuccess;
}

hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
  tick();
  memmove(dst, src, n);
  return hipSuccess;
}

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  tick();
  memmove(dst, src, n);
  return hipSuccess;
}

hipError_t hipMemsetAsync(void* dst, int v, size_t n, hipStream_t) {
  tick();
  memset(dst, v, n);
  return hipSuccess;
}

hipError_t hipGetDevice(int* d) {
  tick();
  *d = 0;
  return hipSuccess;
}
hipError_t hipSetDevice(int) { return api(); }
hipError_t hipGetLastError(void) { return api(); }
hipError_t hipDeviceSynchronize(void) { return api(); }
hipError_t hipStreamSynchronize(hipStream_t) { return api(); }
const char* hipGetErrorString(hipError_t) { return "hip stub error"; }

hipError_t hipEventCreate(hipEvent_t* e) {
  tick();
  *e = reinterpret_cast<hipEvent_t>(new int(0));
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  tick();
  delete reinterpret_cast<int*>(e);
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return api(); }
hipError_t hipStreamCreateWithFlags(hipStream_t* st, unsigned) {
  tick();
  *st = reinterpret_cast<hipStream_t>(new int(0));
  return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t st) {
  tick();
  delete reinterpret_cast<int*>(st);
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned) { return api(); }
hipError_t hipEventSynchronize(hipEvent_t) { return api(); }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  tick();
  *ms = g_elapsed_decreasing ? (g_elapsed *= 0.9f) : 0.25f;
  return hipSuccess;
}

namespace elasto {
hipError_t launch_conv_bf16(const ConvArgs&, hipStream_t) { return launch(); }
hipError_t launch_gemm_bf16(Epi, const GemmArgs&, hipStream_t) { return launch(); }
hipError_t launch_gemm_f32(Epi, const GemmArgs&, hipStream_t) { return launch(); }
hipError_t launch_layernorm_bf16(const void*, int64_t, const float*, int, void*, int64_t, int,
                                 const float*, const float*, float, hipStream_t) {
  return launch();
}
hipError_t launch_layernorm_f32(const void*, int64_t, void*, int64_t, int, const float*,
                                const float*, float, hipStream_t) {
  return launch();
}
hipError_t launch_attention_bf16(const AttnArgs&, hipStream_t) { return launch(); }
hipError_t launch_attention_f32(const AttnArgs&, hipStream_t) { return launch(); }
hipError_t launch_attention_bwd_bf16(const AttnBwdArgs&, hipStream_t) { return launch(); }
hipError_t launch_transpose_bf16(const void*, int64_t, int64_t, int, int, void*, int64_t,
                                 hipStream_t) {
  return launch();
}
hipError_t launch_layernorm_bwd_bf16(const void*, int64_t, const void*, int64_t, const float*,
                                     float, int, int, float*, int64_t, void*, int64_t,
                                     hipStream_t) {
  return launch();
}
hipError_t launch_cross_entropy(const float*, int64_t, const int32_t*, int, int, void*, int64_t,
                                float*, hipStream_t) {
  return launch();
}
hipError_t launch_rowsum_bf16(const void*, int64_t, int, int, float*, hipStream_t) {
  return launch();
}
hipError_t launch_splitk_reduce(const float*, int64_t, int, int, int, int64_t, float*, int64_t,
                                hipStream_t) {
  return launch();
}
int growth_sumsq_parts() { return 64; }
hipError_t launch_growth_norm(const float*, int64_t, float*, const float*, int, float, float*,
                              hipStream_t) {
  return launch();
}
hipError_t launch_growth_update(const GrowthSlice*, int, const float*, float*, void*,
                                const float*, float, hipStream_t) {
  return launch();
}
hipError_t launch_master_init(const void*, int64_t, int64_t, float*, hipStream_t) {
  return launch();
}
hipError_t launch_ln_fold(const void*, int, int, const float*, const float*, const float*,
                          const int*, int, void*, float*, float*, int64_t, hipStream_t) {
  return launch();
}
hipError_t launch_pad_nhwc4(const void*, int, int, int, int, int, void*, hipStream_t) {
  return launch();
}
hipError_t launch_max_pool_3x3_s2(const void*, int, int, int, int, void*, hipStream_t) {
  return launch();
}
hipError_t launch_avg_pool(const void*, int, int, int, void*, hipStream_t) { return launch(); }
hipError_t launch_stem_pool(const void*, int, int, int, const void*, int, const float*, int, void*,
                            hipStream_t) {
  return launch();
}

hipError_t static_scratch(void** ptr, int64_t* bytes) {
  tick();
  if (!g_static) g_static = static_cast<uint8_t*>(aligned_alloc(256, kStaticScratchBytes));
  *ptr = g_static;
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}
}  // namespace elasto

extern "C" void hipstub_release_static(void) {
  free(g_static);
  g_static = nullptr;
}
