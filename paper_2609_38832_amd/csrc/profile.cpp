// Opt-in kernel timing with HIP events (diagnostics; off by default).
//
// When enabled, the launchers time their main kernels of each call with a
// pair of events on the call's stream: either events attached to the kernel
// dispatch itself (prof_pair, launched through hipExtLaunchKernel, so the
// interval is the kernel's own start and end, as a kernel trace records
// it), or events recorded before and after a group of launches (prof_mark).
// Reading the results synchronises on the recorded events.  Not safe for concurrent use from
// several host threads; enabling allocates events, so it is meant for
// benchmarks, not for code that must not allocate.
#include <hip/hip_runtime.h>

#include <cstring>
#include <string>
#include <vector>

#include "internal.h"

namespace namoh {
namespace {

struct Section {
  std::string name;
  std::vector<hipEvent_t> start, stop;
  int used = 0;
};

struct Profiler {
  bool on = false;
  int capacity = 0;
  std::vector<Section> sections;

  Section* find(const char* name, bool create) {
    for (auto& s : sections)
      if (s.name == name) return &s;
    if (!create) return nullptr;
    sections.emplace_back();
    Section& s = sections.back();
    s.name = name;
    s.start.resize(capacity, nullptr);
    s.stop.resize(capacity, nullptr);
    return &s;
  }

  void clear() {
    for (auto& s : sections) {
      for (auto e : s.start) if (e) (void)hipEventDestroy(e);
      for (auto e : s.stop) if (e) (void)hipEventDestroy(e);
    }
    sections.clear();
  }
};

Profiler g_prof;

}  // namespace

void prof_mark(const char* section, bool begin, hipStream_t st) {
  if (!g_prof.on) return;
  Section* s = g_prof.find(section, true);
  if (begin) {
    if (s->used >= g_prof.capacity) return;
    hipEvent_t& e = s->start[s->used];
    if (!e && hipEventCreate(&e) != hipSuccess) { e = nullptr; return; }
    (void)hipEventRecord(e, st);
  } else {
    if (s->used >= g_prof.capacity || !s->start[s->used]) return;
    hipEvent_t& e = s->stop[s->used];
    if (!e && hipEventCreate(&e) != hipSuccess) { e = nullptr; return; }
    (void)hipEventRecord(e, st);
    ++s->used;
  }
}

bool prof_pair(const char* section, hipEvent_t* start, hipEvent_t* stop) {
  *start = *stop = nullptr;
  if (!g_prof.on) return false;
  Section* s = g_prof.find(section, true);
  if (s->used >= g_prof.capacity) return false;
  hipEvent_t& a = s->start[s->used];
  hipEvent_t& b = s->stop[s->used];
  if (!a && hipEventCreate(&a) != hipSuccess) { a = nullptr; return false; }
  if (!b && hipEventCreate(&b) != hipSuccess) { b = nullptr; return false; }
  *start = a;
  *stop = b;
  ++s->used;
  return true;
}

}  // namespace namoh

extern "C" {

// Starts (capacity > 0) or stops (capacity == 0) timing; clears old records.
int namoh_profile_enable(int capacity) {
  namoh::g_prof.clear();
  namoh::g_prof.on = capacity > 0;
  namoh::g_prof.capacity = capacity > 0 ? capacity : 0;
  return 0;
}

// Total milliseconds and number of timed launches of one section
// ("attn", "pack", "decode_attn", ...).  Returns 0, or -1 if unknown.
int namoh_profile_read(const char* section, double* total_ms, int* count) {
  *total_ms = 0.0;
  *count = 0;
  for (auto& s : namoh::g_prof.sections) {
    if (s.name != section) continue;
    for (int i = 0; i < s.used; ++i) {
      if (hipEventSynchronize(s.stop[i]) != hipSuccess) return -1;
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, s.start[i], s.stop[i]) != hipSuccess) return -1;
      *total_ms += ms;
    }
    *count = s.used;
    return 0;
  }
  return -1;
}

}  // extern "C"
