// Launch hooks of the profiling build (libphsa_prof.so): every kernel launch
// is bracketed by two HIP events on its stream, so that a benchmark can read
// the duration of each kernel.  These definitions replace the empty ones of
// api.hip when this file is linked in; libphsa.so does not contain it.
#include <string.h>

#include <mutex>
#include <vector>

#include "phsa_prof.h"
#include "../launch.h"

namespace phsa {

namespace {

struct Rec {
  const char *name;  // a string literal of the launcher
  hipEvent_t a, b;
};

struct State {
  std::mutex mu;
  bool on = false;
  std::vector<Rec> recs;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pool;
  Rec open{nullptr, nullptr, nullptr};
};

State &state() {
  static State s;
  return s;
}

}  // namespace

void timing_begin(const char *name, hipStream_t s) {
  State &st = state();
  std::lock_guard<std::mutex> lock(st.mu);
  if (!st.on) return;
  std::pair<hipEvent_t, hipEvent_t> ev{nullptr, nullptr};
  if (!st.pool.empty()) {
    ev = st.pool.back();
    st.pool.pop_back();
  } else if (hipEventCreate(&ev.first) != hipSuccess || hipEventCreate(&ev.second) != hipSuccess) {
    return;
  }
  st.open = Rec{name, ev.first, ev.second};
  (void)hipEventRecord(ev.first, s);
}

void timing_end(hipStream_t s) {
  State &st = state();
  std::lock_guard<std::mutex> lock(st.mu);
  if (!st.on || !st.open.name) return;
  (void)hipEventRecord(st.open.b, s);
  st.recs.push_back(st.open);
  st.open = Rec{nullptr, nullptr, nullptr};
}

}  // namespace phsa

using namespace phsa;

extern "C" {

phsa_status phsa_prof_enable(int32_t enable) {
  State &st = state();
  std::lock_guard<std::mutex> lock(st.mu);
  st.on = enable != 0;
  return PHSA_OK;
}

int32_t phsa_prof_durations(const char *name, float *ms, int32_t cap) {
  State &st = state();
  std::lock_guard<std::mutex> lock(st.mu);
  int32_t n = 0;
  if (!name) return 0;
  for (const Rec &r : st.recs) {
    if (strcmp(name, r.name) != 0) continue;
    float t = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) t = -1.f;
    if (ms && n < cap) ms[n] = t;
    ++n;
  }
  return n;
}

void phsa_prof_reset(void) {
  State &st = state();
  std::lock_guard<std::mutex> lock(st.mu);
  for (const Rec &r : st.recs) st.pool.emplace_back(r.a, r.b);
  st.recs.clear();
}

}  // extern "C"
