// Per-kernel timing for the library's own launches (off unless started).
//
// The paper profiles per-operator latency to feed its predictors (section 4.1,
// section 5 "Profiling module"); this is the single-GPU, per-kernel analogue.
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "aflex.h"
#include "profile.h"

namespace aflex {
namespace {

struct Rec {
  std::string name;
  hipEvent_t start;
  hipEvent_t stop;
};

std::mutex g_mu;
std::atomic<bool> g_active{false};
std::string g_filter;  // comma-separated kernel names; empty = all
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_free;
std::map<std::string, size_t> g_open;  // name -> index of the record awaiting its stop event

hipEvent_t take_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

bool profile_wants(const char* name) {
  if (!g_active.load(std::memory_order_relaxed)) return false;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_filter.empty()) return true;
  const std::string n(name);
  size_t pos = 0;
  while (pos <= g_filter.size()) {
    size_t end = g_filter.find(',', pos);
    if (end == std::string::npos) end = g_filter.size();
    if (g_filter.compare(pos, end - pos, n) == 0) return true;
    pos = end + 1;
  }
  return false;
}

void profile_mark(const char* name, hipStream_t stream, bool begin) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (begin) {
    Rec r{name, take_event(), nullptr};
    if (r.start && hipEventRecord(r.start, stream) != hipSuccess) {
      g_free.push_back(r.start);
      r.start = nullptr;
    }
    g_open[r.name] = g_recs.size();
    g_recs.push_back(r);
  } else {
    auto it = g_open.find(name);
    if (it == g_open.end()) return;
    Rec& r = g_recs[it->second];
    r.stop = take_event();
    if (r.stop && hipEventRecord(r.stop, stream) != hipSuccess) {
      g_free.push_back(r.stop);
      r.stop = nullptr;
    }
    g_open.erase(it);
  }
}

// Destroys every event the profiler holds (records and the free list) and
// ends an active session. The caller guarantees that no recorded event is
// still pending on a stream.
hipError_t profile_release() {
  g_active.store(false);
  std::lock_guard<std::mutex> lock(g_mu);
  hipError_t first = hipSuccess;
  auto destroy = [&](hipEvent_t e) {
    if (!e) return;
    const hipError_t r = hipEventDestroy(e);
    if (first == hipSuccess) first = r;
  };
  for (auto& r : g_recs) {
    destroy(r.start);
    destroy(r.stop);
  }
  for (hipEvent_t e : g_free) destroy(e);
  g_recs.clear();
  g_free.clear();
  g_open.clear();
  return first;
}

}  // namespace aflex

extern "C" {

aflex_status aflex_profile_start(const char* kernels) {
  std::lock_guard<std::mutex> lock(aflex::g_mu);
  for (auto& r : aflex::g_recs) {
    if (r.start) aflex::g_free.push_back(r.start);
    if (r.stop) aflex::g_free.push_back(r.stop);
  }
  aflex::g_recs.clear();
  aflex::g_open.clear();
  aflex::g_filter = kernels ? kernels : "";
  aflex::g_active.store(true);
  return AFLEX_OK;
}

aflex_status aflex_profile_stop(char* report, size_t len) {
  aflex::g_active.store(false);
  std::lock_guard<std::mutex> lock(aflex::g_mu);
  struct Acc {
    long n = 0;
    double total = 0, mn = 1e30, mx = 0;
  };
  std::map<std::string, Acc> acc;
  aflex_status st = AFLEX_OK;
  for (auto& r : aflex::g_recs) {
    if (!r.start || !r.stop) continue;
    float ms = 0.f;
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      st = AFLEX_ERR_HIP;
      continue;
    }
    Acc& a = acc[r.name];
    a.n += 1;
    a.total += ms;
    a.mn = ms < a.mn ? ms : a.mn;
    a.mx = ms > a.mx ? ms : a.mx;
  }
  for (auto& r : aflex::g_recs) {
    if (r.start) aflex::g_free.push_back(r.start);
    if (r.stop) aflex::g_free.push_back(r.stop);
  }
  aflex::g_recs.clear();
  aflex::g_open.clear();
  if (report && len) {
    size_t used = 0;
    report[0] = 0;
    for (auto& kv : acc) {
      int w = snprintf(report + used, len - used, "%s %ld %.6f %.6f %.6f\n", kv.first.c_str(), kv.second.n,
                       kv.second.total, kv.second.mn, kv.second.mx);
      if (w < 0 || (size_t)w >= len - used) break;
      used += (size_t)w;
    }
  }
  return st;
}

}  // extern "C"
