// Optional per-kernel timing with HIP events (diagnostics for benchmarks).
//
// Every kernel of the library is launched through launch() below.  While
// timing is enabled, the launch carries a start and a stop event that the
// runtime sets at the kernel's own start and end (hipExtLaunchKernel), so the
// measured time is the kernel's, without separate event packets on the
// stream.  Events are host-side runtime objects taken from a pool that grows
// on demand; no device memory is allocated.  This timing pool is the
// library's only mutable global state; it is not thread safe and is meant for
// single-threaded benchmark drivers.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

namespace kda {

// Events for the next launch of `kind` (both null while timing is off).
struct ProfEvents {
  hipEvent_t start, stop;
};
ProfEvents prof_events(const char* kind);

// Device counter of fit work (row-segment x candidate evaluations) while
// profiling is enabled, else nullptr.
unsigned long long* prof_counter();

// Launch kernel k on stream st (timed under `kind` while timing is on).
template <typename... KArgs, typename... Args>
hipError_t launch(const char* kind, void (*k)(KArgs...), dim3 grid, dim3 block, size_t lds,
                  hipStream_t st, Args... args) {
  const ProfEvents ev = prof_events(kind);
  hipExtLaunchKernelGGL(k, grid, block, (std::uint32_t)lds, st, ev.start, ev.stop, 0u,
                        static_cast<KArgs>(args)...);
  return hipGetLastError();
}

}  // namespace kda
