// Launch timing for measurement: while a class is armed, each launcher of that
// class opens a record (prof_begin) whose start/stop events the next launch of
// the thread binds to its dispatch (jg::launch), then closes it (prof_end).
// Events come from a pool that grows on first use and is reused afterwards.
#include <mutex>
#include <vector>

#include "../../include/jagg.h"
#include "prof.h"

namespace jg {

namespace {
struct Rec { hipEvent_t a, b; double work; bool bound; };
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
thread_local int t_pending = -1;
}  // namespace

bool prof_armed() { return P().cls != PROF_NONE; }

int prof_begin(int cls) {
  Prof& p = P();
  if (p.cls == PROF_NONE || cls != p.cls) return -1;
  std::lock_guard<std::mutex> g(p.mu);
  Rec r{take_event(p), take_event(p), 0.0, false};
  if (!r.a || !r.b) return -1;
  p.recs.push_back(r);
  t_pending = (int)p.recs.size() - 1;
  return t_pending;
}

bool prof_take(hipEvent_t* start, hipEvent_t* stop) {
  if (t_pending < 0) return false;
  Prof& p = P();
  std::lock_guard<std::mutex> g(p.mu);
  if (t_pending >= (int)p.recs.size()) { t_pending = -1; return false; }
  Rec& r = p.recs[t_pending];
  *start = r.a;
  *stop = r.b;
  r.bound = true;
  t_pending = -1;
  return true;
}

void prof_end(int idx, double work) {
  if (idx < 0) return;
  Prof& p = P();
  std::lock_guard<std::mutex> g(p.mu);
  if (t_pending == idx) t_pending = -1;  // nothing was launched
  if (idx < (int)p.recs.size()) p.recs[idx].work = work;
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
  jg::t_pending = -1;
  return JAGG_OK;
}

jagg_status jagg_prof_end(long* launches, double* total_ms, double* total_work) {
  auto& p = jg::P();
  std::lock_guard<std::mutex> g(p.mu);
  double ms = 0.0, work = 0.0;
  long n = 0;
  jagg_status st = JAGG_OK;
  for (auto& r : p.recs) {
    if (!r.bound) continue;  // the launcher returned before launching
    float t = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) {
      jg::set_error("jagg_prof_end: a launch's timing events failed");
      st = JAGG_EDEVICE;
      break;
    }
    ms += t;
    work += r.work;
    ++n;
  }
  if (st == JAGG_OK) {
    if (launches) *launches = n;
    if (total_ms) *total_ms = ms;
    if (total_work) *total_work = work;
  }
  p.cls = jg::PROF_NONE;
  p.recs.clear();
  p.used = 0;
  jg::t_pending = -1;
  return st;
}

}  // extern "C"
