// Per-kernel event timing (see kda_profile.hpp).
#include "kda_profile.hpp"

#include <cstring>
#include <string>
#include <vector>

#include "../../include/kda.h"

namespace kda {
namespace {

struct Mark {
  const char* kind;
  hipEvent_t start, stop;
};

bool g_on = false;          // per-kernel events
bool g_count = false;       // quantiser work counter
std::vector<Mark> g_marks;      // recorded since the last read
std::vector<hipEvent_t> g_pool; // spare events
unsigned long long* g_counter = nullptr;   // device memory, 8 bytes

hipEvent_t take() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

ProfEvents prof_events(const char* kind) {
  if (!g_on) return {nullptr, nullptr};
  hipEvent_t a = take(), b = take();
  if (!a || !b) return {nullptr, nullptr};
  g_marks.push_back({kind, a, b});
  return {a, b};
}

unsigned long long* prof_counter() { return g_count ? g_counter : nullptr; }

}  // namespace kda

extern "C" {

int kda_profile_enable(int flags) {
  if ((flags & KDA_PROFILE_COUNTERS) && kda::g_counter == nullptr) {
    if (hipMalloc(&kda::g_counter, sizeof(unsigned long long)) != hipSuccess) return KDA_ERR_HIP;
    if (hipMemset(kda::g_counter, 0, sizeof(unsigned long long)) != hipSuccess) return KDA_ERR_HIP;
  }
  kda::g_on = (flags & KDA_PROFILE_EVENTS) != 0;
  kda::g_count = (flags & KDA_PROFILE_COUNTERS) != 0;
  return KDA_OK;
}

int kda_profile_counters(unsigned long long* fit_evals) {
  if (!fit_evals) return KDA_ERR_ARG;
  *fit_evals = 0;
  if (kda::g_counter == nullptr) return KDA_OK;
  if (hipDeviceSynchronize() != hipSuccess) return KDA_ERR_HIP;
  if (hipMemcpy(fit_evals, kda::g_counter, sizeof(unsigned long long), hipMemcpyDeviceToHost) != hipSuccess)
    return KDA_ERR_HIP;
  if (hipMemset(kda::g_counter, 0, sizeof(unsigned long long)) != hipSuccess) return KDA_ERR_HIP;
  return KDA_OK;
}

int kda_profile_read(int max_kinds, const char** kinds, double* ms, int* counts, int* n_kinds) {
  using namespace kda;
  if (max_kinds < 0 || !n_kinds) return KDA_ERR_ARG;
  int n = 0;
  if (!g_marks.empty() && hipEventSynchronize(g_marks.back().stop) != hipSuccess) return KDA_ERR_HIP;
  std::vector<std::string> names;
  std::vector<double> tot;
  std::vector<int> cnt;
  std::vector<const char*> ptrs;
  for (const Mark& m : g_marks) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, m.start, m.stop) != hipSuccess) return KDA_ERR_HIP;
    int idx = -1;
    for (size_t i = 0; i < names.size(); ++i)
      if (names[i] == m.kind) idx = (int)i;
    if (idx < 0) {
      names.push_back(m.kind);
      ptrs.push_back(m.kind);
      tot.push_back(0.0);
      cnt.push_back(0);
      idx = (int)names.size() - 1;
    }
    tot[idx] += t;
    cnt[idx] += 1;
    g_pool.push_back(m.start);
    g_pool.push_back(m.stop);
  }
  g_marks.clear();
  n = (int)names.size();
  for (int i = 0; i < n && i < max_kinds; ++i) {
    if (kinds) kinds[i] = ptrs[i];   // static strings of the library
    if (ms) ms[i] = tot[i];
    if (counts) counts[i] = cnt[i];
  }
  *n_kinds = n;
  return KDA_OK;
}

}  // extern "C"
