// Thread-local error text and the optional per-launch event timing used for
// measurement (orbit_timing_*).
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace orbit {

static thread_local char g_err[512] = {0};

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}
void clear_error() { g_err[0] = 0; }

// ---------------------------------------------------------------------------
// timing
// ---------------------------------------------------------------------------
namespace {
constexpr int kMaxRecords = 1 << 15;
struct Record {
  const char* name;
  double flops, bytes;
  hipEvent_t start, stop;
};
struct Timing {
  bool on = false;
  std::vector<hipEvent_t> pool;  // 2 * kMaxRecords events, created on first enable
  std::vector<Record> recs;
  int open = -1;
  std::vector<std::string> names;
  std::string filter;
};
Timing& T() {
  static Timing t;
  return t;
}
}  // namespace

bool timing_on() { return T().on; }

void timing_begin(hipStream_t s, const KernelInfo& k) {
  Timing& t = T();
  t.open = -1;
  if ((int)t.recs.size() >= kMaxRecords) return;
  if (!t.filter.empty() && strncmp(k.name, t.filter.c_str(), t.filter.size()) != 0) return;
  const int i = (int)t.recs.size();
  Record r{k.name, k.flops, k.bytes, t.pool[2 * i], t.pool[2 * i + 1]};
  if (hipEventRecord(r.start, s) != hipSuccess) return;
  t.recs.push_back(r);
  t.open = i;
}

void timing_end(hipStream_t s) {
  Timing& t = T();
  if (t.open < 0) return;
  (void)hipEventRecord(t.recs[t.open].stop, s);
  t.open = -1;
}

}  // namespace orbit

using namespace orbit;

extern "C" {

const char* orbit_last_error(void) { return g_err; }

const char* orbit_status_string(orbit_status s) {
  switch (s) {
    case ORBIT_OK: return "ok";
    case ORBIT_E_ARG: return "invalid argument";
    case ORBIT_E_UNSUPPORTED: return "unsupported";
    case ORBIT_E_DEVICE: return "device error";
  }
  return "unknown status";
}

int orbit_abi_version(void) { return ORBIT_ABI_VERSION; }

orbit_status orbit_timing_enable(int on) {
  Timing& t = T();
  if (on) {
    if (t.pool.empty()) {
      t.pool.resize(2 * kMaxRecords);
      for (auto& e : t.pool) {
        if (hipEventCreate(&e) != hipSuccess) {
          set_error("orbit_timing_enable: hipEventCreate failed");
          t.pool.clear();
          return ORBIT_E_DEVICE;
        }
      }
    }
    t.recs.clear();
    t.names.clear();
  }
  t.on = on != 0;
  return ORBIT_OK;
}

orbit_status orbit_timing_filter(const char* prefix) {
  T().filter = prefix ? prefix : "";
  return ORBIT_OK;
}

orbit_status orbit_timing_summary(const char* prefix, int64_t* launches, double* total_ms,
                                  double* flops, double* bytes) {
  Timing& t = T();
  int64_t n = 0;
  double ms = 0, fl = 0, by = 0;
  const size_t plen = prefix ? strlen(prefix) : 0;
  t.names.clear();
  for (const Record& r : t.recs) {
    if (std::find(t.names.begin(), t.names.end(), std::string(r.name)) == t.names.end())
      t.names.emplace_back(r.name);
    if (plen && strncmp(r.name, prefix, plen) != 0) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess) {
      set_error("orbit_timing_summary: hipEventSynchronize failed");
      return ORBIT_E_DEVICE;
    }
    float e = 0.f;
    if (hipEventElapsedTime(&e, r.start, r.stop) != hipSuccess) {
      set_error("orbit_timing_summary: hipEventElapsedTime failed");
      return ORBIT_E_DEVICE;
    }
    ++n;
    ms += e;
    fl += r.flops;
    by += r.bytes;
  }
  if (launches) *launches = n;
  if (total_ms) *total_ms = ms;
  if (flops) *flops = fl;
  if (bytes) *bytes = by;
  return ORBIT_OK;
}

const char* orbit_timing_kernel_name(int i) {
  Timing& t = T();
  if (t.names.empty()) {
    for (const Record& r : t.recs)
      if (std::find(t.names.begin(), t.names.end(), std::string(r.name)) == t.names.end())
        t.names.emplace_back(r.name);
  }
  if (i < 0 || i >= (int)t.names.size()) return nullptr;
  return t.names[i].c_str();
}

}  // extern "C"
