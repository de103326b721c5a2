// Library-wide C entry points that launch nothing, and the opt-in kernel
// timing instrumentation.
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

namespace moe {
namespace {

struct Rec {
  const char* name;
  hipEvent_t start, stop;
};

std::mutex g_mu;
bool g_on = false;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  // timing only: no system-scope fence (cache writeback and invalidation)
  // when the event completes, so the instrumentation does not slow the
  // kernels that follow it
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

bool timing_enabled() {
  std::lock_guard<std::mutex> lk(g_mu);
  return g_on;
}

void timing_record(const char* name, hipStream_t s, bool start) {
  std::lock_guard<std::mutex> lk(g_mu);
  hipEvent_t e = take_event();
  if (!e) return;
  if (hipEventRecord(e, s) != hipSuccess) {
    g_pool.push_back(e);
    return;
  }
  if (start) {
    g_recs.push_back(Rec{name, e, nullptr});
  } else {
    // close the most recent open record of this name
    for (auto it = g_recs.rbegin(); it != g_recs.rend(); ++it) {
      if (it->name == name && it->stop == nullptr) {
        it->stop = e;
        return;
      }
    }
    g_pool.push_back(e);
  }
}

}  // namespace moe

using namespace moe;


extern "C" const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "MOE_OK";
    case MOE_EINVAL: return "MOE_EINVAL: invalid argument";
    case MOE_EUNSUPPORTED: return "MOE_EUNSUPPORTED: unsupported request";
    case MOE_EHIP: return "MOE_EHIP: HIP launch failed";
    case MOE_EWORKSPACE: return "MOE_EWORKSPACE: workspace missing or too small";
    default: return "unknown moe_status";
  }
}

extern "C" int moe_abi_version(void) { return 7; }

extern "C" moe_status moe_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_on = on != 0;
  return MOE_OK;
}

extern "C" int moe_timing_report(char* buf, size_t len) {
  std::vector<Rec> recs;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    recs.swap(g_recs);
  }
  std::map<std::string, std::pair<long, double>> agg;  // name -> (launches, total ms)
  std::vector<std::string> order;
  for (const Rec& r : recs) {
    if (!r.stop) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess) continue;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) continue;
    auto it = agg.find(r.name);
    if (it == agg.end()) {
      order.push_back(r.name);
      agg[r.name] = {1, ms};
    } else {
      it->second.first += 1;
      it->second.second += ms;
    }
  }
  {
    std::lock_guard<std::mutex> lk(g_mu);
    for (const Rec& r : recs) {
      g_pool.push_back(r.start);
      if (r.stop) g_pool.push_back(r.stop);
    }
  }
  std::string out;
  for (const std::string& n : order) {
    char line[256];
    snprintf(line, sizeof(line), "%s %ld %.6f\n", n.c_str(), agg[n].first, agg[n].second);
    out += line;
  }
  if (buf && len > 0) {
    size_t n = out.size() < len - 1 ? out.size() : len - 1;
    std::memcpy(buf, out.data(), n);
    buf[n] = 0;
  }
  return static_cast<int>(order.size());
}
