// Per-kernel-class event timing (see timing.h and eogp_timing_* in eogp.h).
#include "timing.h"

#include <mutex>
#include <vector>

namespace eogp {
namespace timing {
namespace {

struct Rec {
  hipEvent_t a = nullptr, b = nullptr;
  int cls = 0;
  bool closed = false;
};

std::mutex mu;
bool on = false;
std::vector<Rec> recs;
std::vector<hipEvent_t> pool;

hipEvent_t take() {
  if (!pool.empty()) {
    hipEvent_t e = pool.back();
    pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

bool enabled() {
  std::lock_guard<std::mutex> g(mu);
  return on;
}

int begin(int cls, hipStream_t s) {
  std::lock_guard<std::mutex> g(mu);
  if (!on) return -1;
  Rec r;
  r.a = take();
  r.b = take();
  r.cls = cls;
  if (!r.a || !r.b) return -1;
  if (hipEventRecord(r.a, s) != hipSuccess) return -1;
  recs.push_back(r);
  return (int)recs.size() - 1;
}

void end(int slot, hipStream_t s) {
  if (slot < 0) return;
  std::lock_guard<std::mutex> g(mu);
  if (slot >= (int)recs.size()) return;
  if (hipEventRecord(recs[slot].b, s) == hipSuccess) recs[slot].closed = true;
}

eogp_status read(int cls, double* total_ms, int64_t* launches) {
  std::lock_guard<std::mutex> g(mu);
  double tot = 0.0;
  int64_t n = 0;
  std::vector<Rec> keep;
  for (Rec& r : recs) {
    if (r.cls != cls) {
      keep.push_back(r);
      continue;
    }
    if (r.closed) {
      if (hipEventSynchronize(r.b) != hipSuccess) return check_hip(hipGetLastError(), "timing");
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
        tot += ms;
        ++n;
      }
    }
    pool.push_back(r.a);
    pool.push_back(r.b);
  }
  recs.swap(keep);
  if (total_ms) *total_ms = tot;
  if (launches) *launches = n;
  return EOGP_OK;
}

void set(bool enable) {
  std::lock_guard<std::mutex> g(mu);
  on = enable;
}

}  // namespace timing
}  // namespace eogp

extern "C" {

eogp_status eogp_timing_enable(int32_t enable) {
  eogp::timing::set(enable != 0);
  return EOGP_OK;
}

eogp_status eogp_timing_read(int32_t kernel_class, double* total_ms, int64_t* launches) {
  if (kernel_class < 0 || kernel_class >= EOGP_KT_COUNT)
    return eogp::fail(EOGP_ERR_INVALID, "timing_read: unknown kernel class");
  return eogp::timing::read(kernel_class, total_ms, launches);
}

}  // extern "C"
