// Host-side services of libhg.so: status strings, error detail, device
// property cache and the optional per-kernel timing log.
#include <cstdarg>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "hg_internal.h"

namespace hg {

namespace {
thread_local char g_detail[512] = "";

std::mutex g_cu_mu;
std::map<int, int> g_cus;

struct TimingRec {
  const char* name;
  hipEvent_t a, b;
};
std::mutex g_tmu;
bool g_timing = false;
std::vector<TimingRec> g_recs;
std::vector<hipEvent_t> g_free;

hipEvent_t get_event() {
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

void set_detail(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_detail, sizeof(g_detail), fmt, ap);
  va_end(ap);
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_detail, sizeof(g_detail), fmt, ap);
  va_end(ap);
  return code;
}

int num_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  std::lock_guard<std::mutex> lk(g_cu_mu);
  auto it = g_cus.find(dev);
  if (it != g_cus.end()) return it->second;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  g_cus[dev] = n;
  return n;
}

bool timing_on() { return g_timing; }

void timing_begin(const char* name, hipStream_t s, void** tok) {
  std::lock_guard<std::mutex> lk(g_tmu);
  hipEvent_t a = get_event(), b = get_event();
  if (!a || !b) {
    *tok = nullptr;
    return;
  }
  (void)hipEventRecord(a, s);
  g_recs.push_back(TimingRec{name, a, b});
  *tok = reinterpret_cast<void*>(g_recs.size());
}

void timing_end(void* tok, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_tmu);
  const size_t idx = reinterpret_cast<size_t>(tok);
  if (idx == 0 || idx > g_recs.size()) return;
  (void)hipEventRecord(g_recs[idx - 1].b, s);
}

}  // namespace hg

using namespace hg;

extern "C" const char* hg_status_string(int status) {
  switch (status) {
    case HG_OK: return "HG_OK";
    case HG_ERR_ARG: return "HG_ERR_ARG: invalid argument";
    case HG_ERR_RANGE: return "HG_ERR_RANGE: id out of range";
    case HG_ERR_CAPACITY: return "HG_ERR_CAPACITY: buffer too small";
    case HG_ERR_HIP: return "HG_ERR_HIP: HIP runtime error";
    case HG_ERR_UNSUPPORTED: return "HG_ERR_UNSUPPORTED: not implemented for these arguments";
    default: return "unknown status";
  }
}

extern "C" const char* hg_last_error_detail(void) { return g_detail; }

extern "C" int hg_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = on != 0;
  return HG_OK;
}

extern "C" int hg_timing_collect(char (*names)[64], int64_t* launches, double* total_ms, int cap) {
  std::lock_guard<std::mutex> lk(g_tmu);
  std::vector<std::string> keys;
  std::map<std::string, std::pair<int64_t, double>> agg;
  int status = HG_OK;
  for (auto& r : g_recs) {
    if (hipEventSynchronize(r.b) != hipSuccess) status = HG_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) status = HG_ERR_HIP;
    auto it = agg.find(r.name);
    if (it == agg.end()) {
      keys.push_back(r.name);
      agg[r.name] = {1, (double)ms};
    } else {
      it->second.first += 1;
      it->second.second += ms;
    }
    g_free.push_back(r.a);
    g_free.push_back(r.b);
  }
  g_recs.clear();
  if (status != HG_OK) return fail(status, "timing events failed");
  const int n = (int)keys.size();
  for (int i = 0; i < n && i < cap; ++i) {
    if (names) {
      std::strncpy(names[i], keys[i].c_str(), 63);
      names[i][63] = 0;
    }
    if (launches) launches[i] = agg[keys[i]].first;
    if (total_ms) total_ms[i] = agg[keys[i]].second;
  }
  return n;
}
