#include "timing.h"

#include <cstdio>
#include <map>
#include <mutex>
#include <string>
#include <vector>

namespace garfield {
namespace {

struct Record {
  const char* name;
  hipEvent_t start;
  hipEvent_t stop;
};

std::mutex g_mu;
int g_on = 0;
std::vector<Record> g_records;
std::vector<hipEvent_t> g_free;  // events ready for reuse

hipEvent_t take_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  return e;
}

void drop_records_locked() {
  for (const Record& r : g_records) {
    if (r.start) g_free.push_back(r.start);
    if (r.stop) g_free.push_back(r.stop);
  }
  g_records.clear();
}

}  // namespace

bool timing_enabled() { return __atomic_load_n(&g_on, __ATOMIC_RELAXED) != 0; }

void timing_set(bool on) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_records.empty()) (void)hipDeviceSynchronize();
  drop_records_locked();
  __atomic_store_n(&g_on, on ? 1 : 0, __ATOMIC_RELAXED);
}

LaunchEvents timing_record(const char* name) {
  std::lock_guard<std::mutex> lock(g_mu);
  LaunchEvents ev;
  ev.start = take_event();
  ev.stop = ev.start ? take_event() : nullptr;
  if (!ev.stop) {
    if (ev.start) g_free.push_back(ev.start);
    return LaunchEvents{};
  }
  g_records.push_back(Record{name, ev.start, ev.stop});
  return ev;
}

size_t timing_summary(char* buf, size_t len) {
  std::lock_guard<std::mutex> lock(g_mu);
  std::map<std::string, std::pair<long, double>> acc;
  std::vector<std::string> order;
  for (const Record& r : g_records) {
    if (!r.start || !r.stop) continue;
    (void)hipEventSynchronize(r.stop);
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      (void)hipGetLastError();
      continue;
    }
    auto it = acc.find(r.name);
    if (it == acc.end()) {
      order.push_back(r.name);
      acc[r.name] = {1, ms};
    } else {
      it->second.first += 1;
      it->second.second += ms;
    }
  }
  std::string out;
  char line[160];
  for (const std::string& name : order) {
    std::snprintf(line, sizeof(line), "%s %ld %.6f\n", name.c_str(), acc[name].first,
                  acc[name].second);
    out += line;
  }
  if (buf && len > 0) {
    const size_t n = out.size() < len - 1 ? out.size() : len - 1;
    out.copy(buf, n);
    buf[n] = '\0';
  }
  return out.size();
}

}  // namespace garfield
