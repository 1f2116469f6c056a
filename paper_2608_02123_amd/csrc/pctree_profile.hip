// Optional hipEvent bracketing of the dominant kernel's launches, and the
// diagnostic launch overrides (see include/pctree_profile.h).  Off by
// default; costs one branch per launch.
#include "pctree_profile.h"

#include <mutex>
#include <vector>

#include "pctree_plan.h"

namespace pctree {
namespace {

struct Recorder {
  std::mutex mu;
  bool on = false;
  std::vector<hipEvent_t> pool;  // start/stop pairs, reused across enables
  size_t used = 0;               // events handed out since enabling
  const char* kernel = "";       // name given by the last mark
};

Recorder& rec() {
  static Recorder r;
  return r;
}

hipEvent_t next_event() {
  Recorder& r = rec();
  if (r.used == r.pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    r.pool.push_back(e);
  }
  return r.pool[r.used++];
}

}  // namespace

bool profile_on() { return rec().on; }

void profile_mark(hipStream_t stream, const char* kernel) {
  Recorder& r = rec();
  std::lock_guard<std::mutex> g(r.mu);
  if (!r.on) return;
  r.kernel = kernel;
  hipEvent_t e = next_event();
  if (e) (void)hipEventRecord(e, stream);
}

}  // namespace pctree

using namespace pctree;

extern "C" {

pctree_status pctree_profile_enable(int32_t enable) {
  Recorder& r = rec();
  std::lock_guard<std::mutex> g(r.mu);
  r.on = enable != 0;
  r.used = 0;
  return PCTREE_OK;
}

pctree_status pctree_profile_read(double* total_ms, int64_t* launches, const char** kernel) {
  if (!total_ms || !launches) return PCTREE_ERR_INVALID_ARGUMENT;
  Recorder& r = rec();
  std::lock_guard<std::mutex> g(r.mu);
  double sum = 0.0;
  const size_t pairs = r.used / 2;
  for (size_t i = 0; i < pairs; ++i) {
    float ms = 0.0f;
    if (hipEventSynchronize(r.pool[2 * i + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms, r.pool[2 * i], r.pool[2 * i + 1]) != hipSuccess)
      return PCTREE_ERR_HIP;
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int64_t)pairs;
  if (kernel) *kernel = r.kernel;
  r.used = 0;
  return PCTREE_OK;
}

pctree_status pctree_debug_set(const pctree_debug_config* cfg) {
  DebugConfig d;
  if (cfg) {
    if (cfg->round_slices < 0) return PCTREE_ERR_INVALID_ARGUMENT;
    d.wait_ticks = cfg->wait_ticks < 0 ? -1 : (long long)cfg->wait_ticks;
    d.force_multilaunch = cfg->force_multilaunch != 0;
    d.round_slices = cfg->round_slices;
    d.wide_unbounded = cfg->wide_unbounded != 0;
  }
  debug_config() = d;
  return PCTREE_OK;
}

int32_t pctree_timeline_available(void) { return timeline_built() ? 1 : 0; }

pctree_status pctree_timeline_read(int64_t* out, double* ticks_per_us) {
  static_assert(kTimelineWho == PCTREE_TIMELINE_WHO && kTimelineStages == PCTREE_TIMELINE_STAGES &&
                    kTimelineEvents == PCTREE_TIMELINE_EVENTS,
                "timeline shape");
  static_assert(sizeof(long long) == sizeof(int64_t), "timeline stamps are 64-bit");
  if (!timeline_built()) return PCTREE_ERR_UNSUPPORTED;
  if (!out || !ticks_per_us) return PCTREE_ERR_INVALID_ARGUMENT;
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      khz <= 0)
    return PCTREE_ERR_HIP;
  if (timeline_copy(reinterpret_cast<long long*>(out), true) != hipSuccess) return PCTREE_ERR_HIP;
  *ticks_per_us = khz / 1000.0;
  return PCTREE_OK;
}

}  // extern "C"
