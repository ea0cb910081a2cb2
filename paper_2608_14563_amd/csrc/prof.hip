// Opt-in per-kernel timing with hipEvents on the launch stream (fpo_prof.h).
#include <hip/hip_runtime.h>

#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/fpo_prof.h"
#include "prof.hpp"

namespace fpo {
namespace {

struct Pending {
  std::string name;
  hipEvent_t a, b;
};

struct Registry {
  std::mutex mu;
  bool on = false;
  std::vector<std::string> filter;
  std::vector<Pending> pending;
  std::map<std::string, std::pair<double, int64_t>> totals;
  // the begin event of the launch in flight on this thread
  bool matches(const char* n) const {
    if (filter.empty()) return true;
    for (const auto& f : filter)
      if (f == n) return true;
    return false;
  }
};

Registry& reg() {
  static Registry r;
  return r;
}

thread_local hipEvent_t t_begin = nullptr;
thread_local const char* t_name = nullptr;

}  // namespace

void prof_begin(const char* name, hipStream_t st) {
  Registry& r = reg();
  t_name = nullptr;
  {
    std::lock_guard<std::mutex> g(r.mu);
    if (!r.on || !r.matches(name)) return;
  }
  if (hipEventCreate(&t_begin) != hipSuccess) return;
  if (hipEventRecord(t_begin, st) != hipSuccess) {
    (void)hipEventDestroy(t_begin);
    return;
  }
  t_name = name;
}

void prof_end(hipStream_t st) {
  if (!t_name) return;
  hipEvent_t e;
  if (hipEventCreate(&e) != hipSuccess) {
    (void)hipEventDestroy(t_begin);
    t_name = nullptr;
    return;
  }
  (void)hipEventRecord(e, st);
  Registry& r = reg();
  std::lock_guard<std::mutex> g(r.mu);
  r.pending.push_back({t_name, t_begin, e});
  t_name = nullptr;
}

}  // namespace fpo

extern "C" {

int fpo_prof_enable(const char* filter) {
  auto& r = fpo::reg();
  std::lock_guard<std::mutex> g(r.mu);
  r.filter.clear();
  if (filter && *filter) {
    std::string s(filter);
    size_t p = 0;
    while (p <= s.size()) {
      size_t q = s.find(',', p);
      if (q == std::string::npos) q = s.size();
      if (q > p) r.filter.push_back(s.substr(p, q - p));
      p = q + 1;
    }
  }
  r.on = true;
  return 0;
}

int fpo_prof_disable(void) {
  auto& r = fpo::reg();
  std::lock_guard<std::mutex> g(r.mu);
  r.on = false;
  return 0;
}

int fpo_prof_read(int max_entries, char* names, double* total_ms, int64_t* launches) {
  auto& r = fpo::reg();
  std::lock_guard<std::mutex> g(r.mu);
  int rc = 0;
  for (auto& p : r.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess) rc = -1;
    auto& t = r.totals[p.name];
    t.first += ms;
    t.second += 1;
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  r.pending.clear();
  if (rc < 0) return rc;
  int i = 0;
  for (auto& kv : r.totals) {
    if (i >= max_entries) break;
    if (names) {
      std::strncpy(names + 32 * i, kv.first.c_str(), 31);
      names[32 * i + 31] = 0;
    }
    if (total_ms) total_ms[i] = kv.second.first;
    if (launches) launches[i] = kv.second.second;
    ++i;
  }
  return (int)r.totals.size() < max_entries ? (int)r.totals.size() : max_entries;
}

int fpo_prof_reset(void) {
  auto& r = fpo::reg();
  std::lock_guard<std::mutex> g(r.mu);
  for (auto& p : r.pending) {
    (void)hipEventSynchronize(p.b);
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  r.pending.clear();
  r.totals.clear();
  return 0;
}

}  // extern "C"
