// Counters and fault injection of the host HIP stand-ins (hip_stub.cpp).
#ifndef ELASTO_TESTS_HIP_STUB_H_
#define ELASTO_TESTS_HIP_STUB_H_

#ifdef __cplusplus
extern "C" {
#endif
long hipstub_api_calls(void);         // HIP runtime calls since the last reset
long hipstub_launches(void);          // kernel launches since the last reset
long hipstub_mallocs(void);           // hipMalloc calls since the last reset
long hipstub_live_allocations(void);  // hipMalloc'd blocks not yet freed
void hipstub_reset_counts(void);
void hipstub_fail_malloc_at(long n);  // the n-th hipMalloc from now fails (n >= 0)
void hipstub_release_static(void);
// hipEventElapsedTime: 0.25 ms (off), or a value that falls with every call
// (on), so that each timed candidate looks faster than the one before.
void hipstub_elapsed_decreasing(int on);
#ifdef __cplusplus
}
#endif
#endif
