// Per-launch timing hook (diagnostics).  While a profile is active every
// kernel launch of the library is bracketed by two HIP events recorded on the
// launch's stream, so the caller can read each kernel's duration without an
// external profiler.  Meant for one thread at a time.
#include <mutex>
#include <vector>

#include "common.h"

namespace moe {

namespace {
struct Profile {
  std::mutex mu;
  bool active = false;
  int count = 0;
  std::vector<hipEvent_t> begin, end;
  std::vector<const char*> names;
};
Profile& prof() {
  static Profile p;
  return p;
}
}  // namespace

void prof_before(hipStream_t s, const char* name) {
  Profile& p = prof();
  if (!p.active) return;
  std::lock_guard<std::mutex> g(p.mu);
  if (p.count >= (int)p.begin.size()) return;
  (void)hipEventRecord(p.begin[p.count], s);
  p.names[p.count] = name;
}

void prof_after(hipStream_t s) {
  Profile& p = prof();
  if (!p.active) return;
  std::lock_guard<std::mutex> g(p.mu);
  if (p.count >= (int)p.begin.size()) return;
  (void)hipEventRecord(p.end[p.count], s);
  ++p.count;
}

}  // namespace moe

using namespace moe;

extern "C" moe_status_t moe_profile_begin(int32_t max_launches) {
  Profile& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  if (max_launches < 1) return fail(MOE_ERR_INVALID_ARG, "moe_profile_begin: max_launches=%d", max_launches);
  if ((int)p.begin.size() < max_launches) {
    const int have = (int)p.begin.size();
    p.begin.resize(max_launches);
    p.end.resize(max_launches);
    for (int i = have; i < max_launches; ++i) {
      if (hipEventCreate(&p.begin[i]) != hipSuccess || hipEventCreate(&p.end[i]) != hipSuccess) {
        p.begin.resize(i);
        p.end.resize(i);
        return fail(MOE_ERR_HIP, "moe_profile_begin: hipEventCreate failed");
      }
    }
  }
  p.names.assign(p.begin.size(), nullptr);
  p.count = 0;
  p.active = true;
  return MOE_OK;
}

extern "C" int32_t moe_profile_end(void) {
  Profile& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  p.active = false;
  for (int i = 0; i < p.count; ++i) (void)hipEventSynchronize(p.end[i]);
  return p.count;
}

extern "C" moe_status_t moe_profile_get(int32_t i, float* ms, const char** name) {
  Profile& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  if (i < 0 || i >= p.count || !ms || !name) return fail(MOE_ERR_INVALID_ARG, "moe_profile_get: index %d", i);
  const hipError_t e = hipEventElapsedTime(ms, p.begin[i], p.end[i]);
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "moe_profile_get: %s", hipGetErrorString(e));
  *name = p.names[i];
  return MOE_OK;
}
