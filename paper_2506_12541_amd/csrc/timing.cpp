// Optional per-phase kernel timing: when enabled, each timed phase of the library records
// a pair of HIP events on the stream its kernels are launched on, so a caller can read
// the average device duration of a kernel over a measured region.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "kernels.hpp"

namespace bsa {
namespace {

struct Record {
  std::string name;
  hipEvent_t start, stop;
};

std::mutex g_mu;
bool g_on = false;
std::vector<std::string> g_only;   // phases recorded while on; empty = every phase
std::vector<Record> g_records;
std::vector<hipEvent_t> g_free;

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

bool timing_on() {
  std::lock_guard<std::mutex> lk(g_mu);
  return g_on;
}

void timing_select(const char* phases) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_only.clear();
  if (!phases) return;
  std::string cur;
  for (const char* c = phases;; ++c) {
    if (*c == ',' || *c == '\0') {
      if (!cur.empty()) g_only.push_back(cur);
      cur.clear();
      if (*c == '\0') break;
    } else {
      cur += *c;
    }
  }
}

void timing_set(bool on) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (auto& r : g_records) {
    hipEventSynchronize(r.stop);
    g_free.push_back(r.start);
    g_free.push_back(r.stop);
  }
  g_records.clear();
  g_on = on;
}

int timing_begin(const char* name, hipStream_t st) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on) return -1;
  if (!g_only.empty()) {
    bool hit = false;
    for (const auto& p : g_only) hit = hit || p == name;
    if (!hit) return -1;
  }
  Record r{name, take_event(), take_event()};
  if (!r.start || !r.stop) return -1;
  hipEventRecord(r.start, st);
  g_records.push_back(r);
  return (int)g_records.size() - 1;
}

void timing_end(int id, hipStream_t st) {
  if (id < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (id < (int)g_records.size()) hipEventRecord(g_records[id].stop, st);
}

hipError_t timing_query(const char* name, double* total_ms, int* count) {
  std::lock_guard<std::mutex> lk(g_mu);
  double tot = 0.0;
  int n = 0;
  for (auto& r : g_records) {
    if (r.name != name) continue;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e != hipSuccess) return e;
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) return e;
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *count = n;
  return hipSuccess;
}

}  // namespace bsa
