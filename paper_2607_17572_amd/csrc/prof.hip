// Launch timing for measurement: while a class is armed, the launchers of that
// class bracket each kernel with a pair of HIP events on the launch stream.
// Events come from a pool that grows on first use and is reused afterwards.
#include <mutex>
#include <vector>

#include "../../include/jagg.h"
#include "prof.h"

namespace jg {

namespace {
struct Rec { hipEvent_t a, b; double work; bool ok; };
struct Prof {
  std::mutex mu;
  int cls = PROF_NONE;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<Rec> recs;
};
Prof& P() {
  static Prof p;
  return p;
}
hipEvent_t take_event(Prof& p) {
  if (p.used == p.pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    p.pool.push_back(e);
  }
  return p.pool[p.used++];
}
}  // namespace

bool prof_armed() { return P().cls != PROF_NONE; }

int prof_begin(int cls, hipStream_t s) {
  Prof& p = P();
  if (p.cls == PROF_NONE || cls != p.cls) return -1;
  std::lock_guard<std::mutex> g(p.mu);
  Rec r{take_event(p), take_event(p), 0.0, false};
  if (!r.a || !r.b || hipEventRecord(r.a, s) != hipSuccess) return -1;
  p.recs.push_back(r);
  return (int)p.recs.size() - 1;
}

void prof_end(int idx, hipStream_t s, double work) {
  if (idx < 0) return;
  Prof& p = P();
  std::lock_guard<std::mutex> g(p.mu);
  p.recs[idx].ok = hipEventRecord(p.recs[idx].b, s) == hipSuccess;
  p.recs[idx].work = work;
}

}  // namespace jg

extern "C" {

jagg_status jagg_prof_begin(int cls) {
  auto& p = jg::P();
  std::lock_guard<std::mutex> g(p.mu);
  if (cls < jg::PROF_GEMM_FWD || cls > jg::PROF_UPSTREAM) {
    jg::set_error("jagg_prof_begin: unknown kernel class");
    return JAGG_EINVAL;
  }
  p.cls = cls;
  p.recs.clear();
  p.used = 0;
  return JAGG_OK;
}

jagg_status jagg_prof_end(long* launches, double* total_ms, double* total_work) {
  auto& p = jg::P();
  std::lock_guard<std::mutex> g(p.mu);
  double ms = 0.0, work = 0.0;
  for (auto& r : p.recs) {
    float t = 0.f;
    if (!r.ok || hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) {
      jg::set_error("jagg_prof_end: a launch's timing events failed");
      p.cls = jg::PROF_NONE;
      p.recs.clear();
      p.used = 0;
      return JAGG_EDEVICE;
    }
    ms += t;
    work += r.work;
  }
  if (launches) *launches = (long)p.recs.size();
  if (total_ms) *total_ms = ms;
  if (total_work) *total_work = work;
  p.cls = jg::PROF_NONE;
  p.recs.clear();
  p.used = 0;
  return JAGG_OK;
}

}  // extern "C"
