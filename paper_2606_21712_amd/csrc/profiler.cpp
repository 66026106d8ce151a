// Optional per-kernel timing with HIP events (a benchmarking aid).
//
// When enabled, every kernel the library launches (or only those of one name,
// after moe_profiler_select) is bracketed by a pair of events recorded on the
// launch stream.  Event pairs come from a pool created by moe_profiler_start(),
// so recording adds no allocation to the hot path.  When disabled (the
// default) a launch pays one relaxed atomic load.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/moe.h"
#include "moe_internal.h"

namespace moe {
namespace {

struct Rec {
  const char* name;
  hipEvent_t a, b;
};

std::atomic<bool> g_on{false};
std::mutex g_mu;
std::vector<Rec> g_pool;   // created by start(), destroyed by the next start()
size_t g_used = 0;
std::string g_only;        // record only launches of this name ("" = all)
thread_local Rec* g_open = nullptr;

}  // namespace

void prof_begin(hipStream_t s, const char* name) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_used >= g_pool.size()) return;
  if (!g_only.empty() && std::strcmp(name, g_only.c_str()) != 0) return;
  Rec* r = &g_pool[g_used++];
  r->name = name;
  hipEventRecord(r->a, s);
  g_open = r;
}

void prof_end(hipStream_t s) {
  if (g_open == nullptr) return;
  hipEventRecord(g_open->b, s);
  g_open = nullptr;
}

}  // namespace moe

extern "C" {

moe_status moe_profiler_start(int capacity) {
  using namespace moe;
  if (capacity < 1) return MOE_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lock(g_mu);
  g_on.store(false);
  for (Rec& r : g_pool) {
    hipEventDestroy(r.a);
    hipEventDestroy(r.b);
  }
  g_pool.clear();
  g_used = 0;
  g_pool.resize(size_t(capacity));
  for (Rec& r : g_pool) {
    r.name = "";
    if (hipEventCreate(&r.a) != hipSuccess || hipEventCreate(&r.b) != hipSuccess) return MOE_ERR_HIP;
  }
  g_on.store(true);
  return MOE_OK;
}

moe_status moe_profiler_select(const char* name) {
  std::lock_guard<std::mutex> lock(moe::g_mu);
  moe::g_only = name != nullptr ? name : "";
  return MOE_OK;
}

moe_status moe_profiler_stop(void) {
  moe::g_on.store(false);
  return MOE_OK;
}

int moe_profiler_count(void) {
  std::lock_guard<std::mutex> lock(moe::g_mu);
  return int(moe::g_used);
}

moe_status moe_profiler_record(int i, const char** name, float* ms) {
  using namespace moe;
  std::lock_guard<std::mutex> lock(g_mu);
  if (i < 0 || size_t(i) >= g_used || name == nullptr || ms == nullptr) return MOE_ERR_INVALID_ARGUMENT;
  *name = g_pool[size_t(i)].name;
  if (hipEventElapsedTime(ms, g_pool[size_t(i)].a, g_pool[size_t(i)].b) != hipSuccess) return MOE_ERR_HIP;
  return MOE_OK;
}

}  // extern "C"
