// Optional per-kernel timing: when a kernel class is enabled, every launch of it
// is bracketed by two hipEvents recorded on the launch stream.  Events come from
// a pool that is reused after dc_profile_reset(), so steady-state timing creates
// no events.  Reading waits for the recorded events.
#include <atomic>
#include <mutex>
#include <vector>

#include "internal.h"

namespace dc {

namespace {
struct Record {
  int cls;
  hipEvent_t start, stop;
};
std::atomic<uint32_t> g_mask{0};
std::mutex g_mu;
std::vector<Record> g_records;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
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

ProfScope::ProfScope(KClass c, hipStream_t s) : cls_(int(c)), stream_(s) {
  if (!(g_mask.load(std::memory_order_relaxed) & (1u << cls_))) return;
  std::lock_guard<std::mutex> lk(g_mu);
  start_ = take_event();
  if (start_ && hipEventRecord(start_, s) != hipSuccess) start_ = nullptr;
}

ProfScope::~ProfScope() {
  if (!start_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  hipEvent_t stop = take_event();
  if (stop && hipEventRecord(stop, stream_) == hipSuccess) g_records.push_back({cls_, start_, stop});
}

}  // namespace dc

using namespace dc;

extern "C" {

dc_status dc_profile_enable(uint32_t mask) {
  g_mask.store(mask);
  return DC_OK;
}

dc_status dc_profile_read(int32_t cls, int64_t* launches, double* total_ms) {
  if (cls < 0 || cls >= int(KClass::kCount) || !launches || !total_ms) {
    return DC_ERR_ARG;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  int64_t n = 0;
  double ms = 0.0;
  for (const Record& r : g_records) {
    if (r.cls != cls) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess) return DC_ERR_HIP;
    float t = 0.f;
    if (hipEventElapsedTime(&t, r.start, r.stop) != hipSuccess) return DC_ERR_HIP;
    ms += double(t);
    ++n;
  }
  *launches = n;
  *total_ms = ms;
  return DC_OK;
}

dc_status dc_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (const Record& r : g_records) {
    if (hipEventSynchronize(r.stop) != hipSuccess) return DC_ERR_HIP;
    g_pool.push_back(r.start);
    g_pool.push_back(r.stop);
  }
  g_records.clear();
  return DC_OK;
}

}  // extern "C"
