// Error reporting, version and the event-based kernel profiler.
#include <cstdarg>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "ff_internal.h"

namespace ff {

static thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return FF_OK;
  return fail(FF_EHIP, "%s: %s", what, hipGetErrorString(e));
}

int ensure_smem_limit(const void* kernel, int bytes, std::atomic<uint64_t>& done) {
  int dev = 0;
  FF_CHECK_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(FF_EUNSUPPORTED, "device ordinal %d above 63", dev);
  const uint64_t bit = uint64_t(1) << dev;
  if (done.load(std::memory_order_acquire) & bit) return FF_OK;
  FF_CHECK_HIP(hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes), "kernel LDS limit");
  done.fetch_or(bit, std::memory_order_acq_rel);
  return FF_OK;
}

// ----------------------------------------------------------------- profiler
namespace {
struct Pending {
  const char* name;
  hipEvent_t a, b;
  double flops, bytes;
};
struct Totals {
  int64_t launches = 0;
  double ms = 0, flops = 0, bytes = 0;
};
std::mutex g_mu;
bool g_on = false;
std::string g_filter;   // empty: every kernel
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
std::map<std::string, Totals> g_totals;

hipEvent_t get_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

int drain_locked() {
  int rc = FF_OK;
  for (auto& p : g_pending) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(p.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.a, p.b);
    if (e != hipSuccess && rc == FF_OK) rc = hip_status(e, "profile event");
    Totals& t = g_totals[p.name];
    t.launches += 1;
    t.ms += ms;
    t.flops += p.flops;
    t.bytes += p.bytes;
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
  }
  g_pending.clear();
  return rc;
}
}  // namespace

LaunchScope::LaunchScope(const char* name, hipStream_t s, double flops, double bytes)
    : name_(name), stream_(s), flops_(flops), bytes_(bytes), slot_(-1) {
  if (!name_) return;   // an unprofiled launch (no events, no allocation)
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on) return;
  if (!g_filter.empty() && g_filter != name_) return;
  hipEvent_t a = get_event(), b = get_event();
  if (!a || !b) return;
  if (hipEventRecord(a, stream_) != hipSuccess) return;
  g_pending.push_back({name_, a, b, flops_, bytes_});
  slot_ = static_cast<int>(g_pending.size()) - 1;
}

LaunchScope::~LaunchScope() {
  if (slot_ < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (slot_ < static_cast<int>(g_pending.size())) hipEventRecord(g_pending[slot_].b, stream_);
}

int LaunchScope::status() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(FF_EHIP, "launch of %s: %s", name_ ? name_ : "kernel", hipGetErrorString(e));
  return FF_OK;
}

}  // namespace ff

using namespace ff;

extern "C" {

const char* ff_last_error(void) { return g_err.c_str(); }

const char* ff_version(void) { return "ff 0.1 gfx950"; }

int ff_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_on = on != 0;
  return FF_OK;
}

int ff_profile_filter(const char* name) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_filter = name ? name : "";
  return FF_OK;
}

int ff_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  int rc = drain_locked();
  g_totals.clear();
  return rc;
}

int ff_profile_count(int32_t* n) {
  if (!n) return fail(FF_EINVAL, "ff_profile_count: null output");
  std::lock_guard<std::mutex> lk(g_mu);
  int rc = drain_locked();
  *n = static_cast<int32_t>(g_totals.size());
  return rc;
}

int ff_profile_read(int32_t i, char* name, size_t name_cap, int64_t* launches, double* total_ms,
                    double* flops, double* bytes) {
  std::lock_guard<std::mutex> lk(g_mu);
  int rc = drain_locked();
  if (rc != FF_OK) return rc;
  if (i < 0 || i >= static_cast<int32_t>(g_totals.size()))
    return fail(FF_EINVAL, "ff_profile_read: index %d out of range", i);
  auto it = g_totals.begin();
  std::advance(it, i);
  if (name && name_cap) {
    strncpy(name, it->first.c_str(), name_cap - 1);
    name[name_cap - 1] = 0;
  }
  if (launches) *launches = it->second.launches;
  if (total_ms) *total_ms = it->second.ms;
  if (flops) *flops = it->second.flops;
  if (bytes) *bytes = it->second.bytes;
  return FF_OK;
}

}  // extern "C"
