// Optional per-launch timing for measurement tools.  When enabled, each kernel
// launch of the library whose site name matches the filter is bracketed by two
// HIP events on the launch stream; tav2_profile_report() turns the recorded
// pairs into per-site totals.  Disabled (the default) it costs one relaxed
// atomic load per launch.
#include <atomic>
#include <map>
#include <mutex>
#include <stdio.h>
#include <string.h>
#include <string>
#include <vector>

#include "common.h"
#include "internal.h"

namespace tav2 {
namespace {

std::atomic<bool> g_on{false};
std::mutex g_mu;
std::string g_filter;   // empty = every site
struct Site {
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pairs;
};
std::map<std::string, Site> g_sites;
std::vector<hipEvent_t> g_free;

hipEvent_t take_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  // timing only: no system-scope fence (and its cache writeback) at each record,
  // which would otherwise slow the work around the timed launches
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

ProfScope::ProfScope(const char* name, hipStream_t st) : name_(name), st_(st), start_(nullptr) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_filter.empty() && g_filter != name) return;
  hipEvent_t e = take_event();
  if (!e) return;
  if (hipEventRecord(e, st_) != hipSuccess) {
    g_free.push_back(e);
    return;
  }
  start_ = e;
}

ProfScope::~ProfScope() {
  if (!start_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  hipEvent_t start = static_cast<hipEvent_t>(start_);
  hipEvent_t stop = take_event();
  if (!stop || hipEventRecord(stop, st_) != hipSuccess) {
    g_free.push_back(start);
    if (stop) g_free.push_back(stop);
    return;
  }
  g_sites[name_].pairs.emplace_back(start, stop);
}

}  // namespace tav2

using namespace tav2;

extern "C" {

int32_t tav2_profile_enable(int32_t on, const char* only_site) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_filter = (on && only_site) ? std::string(only_site) : std::string();
  g_on.store(on != 0, std::memory_order_relaxed);
  return TAV2_OK;
}

int64_t tav2_profile_report(char* buf, size_t buf_bytes) {
  std::lock_guard<std::mutex> lk(g_mu);
  std::string text;
  for (auto& kv : g_sites) {
    double total_ms = 0.0;
    long count = 0;
    for (auto& pr : kv.second.pairs) {
      float ms = 0.f;
      if (hipEventSynchronize(pr.second) == hipSuccess &&
          hipEventElapsedTime(&ms, pr.first, pr.second) == hipSuccess) {
        total_ms += ms;
        ++count;
      }
      g_free.push_back(pr.first);
      g_free.push_back(pr.second);
    }
    if (count == 0) continue;
    char line[256];
    snprintf(line, sizeof line, "%s %ld %.6f\n", kv.first.c_str(), count, total_ms);
    text += line;
  }
  g_sites.clear();
  if (buf && buf_bytes > 0) {
    const size_t n = text.size() < buf_bytes - 1 ? text.size() : buf_bytes - 1;
    memcpy(buf, text.data(), n);
    buf[n] = '\0';
  }
  return int64_t(text.size());
}

}  // extern "C"
