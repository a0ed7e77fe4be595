// Optional per-kernel timing with HIP events (diagnostics for benchmarks).
//
// While enabled, every kernel a libkda call enqueues is bracketed by two
// events recorded on the call's stream.  Events are host-side runtime objects
// taken from a pool that grows on demand; no device memory is allocated.
// This timing pool is the library's only mutable global state; it is not
// thread safe and is meant for single-threaded benchmark drivers.
#pragma once

#include <hip/hip_runtime.h>

namespace kda {

void prof_begin(const char* kind, hipStream_t st);
void prof_end(hipStream_t st);

// Device counter of fit work (row-segment x candidate evaluations) while
// profiling is enabled, else nullptr.
unsigned long long* prof_counter();

struct ProfScope {
  hipStream_t st;
  ProfScope(const char* kind, hipStream_t s) : st(s) { prof_begin(kind, s); }
  ~ProfScope() { prof_end(st); }
};

}  // namespace kda
