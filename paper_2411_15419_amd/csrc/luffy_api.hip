// Status strings, error reporting and ABI version.
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <utility>
#include <vector>

#include "luffy_common.h"

namespace luffy {

static thread_local char g_last_error[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
}

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("%s: %s", what, hipGetErrorString(e));
    return LUFFY_E_HIP;
  }
  return LUFFY_OK;
}

int persistent_grid() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int cus = 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 256;
    cached[dev] = cus;
  }
  return cached[dev];
}

// ---------------------------------------------------------------- profiling
namespace {
std::atomic<bool> g_prof_on{false};
std::mutex g_prof_mu;
char g_prof_name[64] = "";
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_prof_done;
std::vector<hipEvent_t> g_prof_pool;

hipEvent_t take_event() {
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

bool profile_begin(const char* name, hipEvent_t* start, hipEvent_t* stop) {
  if (!g_prof_on.load(std::memory_order_relaxed)) return false;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (std::strcmp(name, g_prof_name) != 0) return false;
  *start = take_event();
  *stop = take_event();
  if (*start && *stop) return true;
  if (*start) g_prof_pool.push_back(*start);
  if (*stop) g_prof_pool.push_back(*stop);
  return false;
}

void profile_end(hipEvent_t start, hipEvent_t stop) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_done.emplace_back(start, stop);
}

}  // namespace luffy

extern "C" int luffy_profile_kernel(const char* name) {
  using namespace luffy;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!name || !*name) {
    g_prof_name[0] = 0;
    g_prof_on.store(false);
    return LUFFY_OK;
  }
  if (std::strlen(name) >= sizeof(g_prof_name))
    return fail(LUFFY_E_INVALID, "luffy_profile_kernel: name too long");
  std::strcpy(g_prof_name, name);
  while (g_prof_pool.size() < 256) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return fail(LUFFY_E_HIP, "luffy_profile_kernel: hipEventCreate");
    g_prof_pool.push_back(e);
  }
  g_prof_on.store(true);
  return LUFFY_OK;
}

extern "C" int luffy_profile_read(double* total_ms, int* launches) {
  using namespace luffy;
  if (!total_ms || !launches) return fail(LUFFY_E_INVALID, "luffy_profile_read: null pointer");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  double sum = 0.0;
  int n = 0;
  int status = LUFFY_OK;
  for (auto& pr : g_prof_done) {
    float ms = 0.f;
    if (hipEventSynchronize(pr.second) != hipSuccess ||
        hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess) {
      status = fail(LUFFY_E_HIP, "luffy_profile_read: event query failed");
    } else {
      sum += ms;
      ++n;
    }
    g_prof_pool.push_back(pr.first);
    g_prof_pool.push_back(pr.second);
  }
  g_prof_done.clear();
  *total_ms = sum;
  *launches = n;
  return status;
}

// Eq. 2 of Sec. 5.2, in double precision on the host.
extern "C" int luffy_adaptive_threshold(double l_ini, double l_prev, double* h_out) {
  if (!h_out) return luffy::fail(LUFFY_E_INVALID, "luffy_adaptive_threshold: h_out is null");
  if (!std::isfinite(l_ini) || l_ini == 0.0)
    return luffy::fail(LUFFY_E_INVALID, "luffy_adaptive_threshold: l_ini=%g must be finite and non-zero", l_ini);
  if (!std::isfinite(l_prev))
    return luffy::fail(LUFFY_E_INVALID, "luffy_adaptive_threshold: l_prev=%g must be finite", l_prev);
  const double l_norm = (l_ini - l_prev) / l_ini;
  *h_out = 1.0 / (1.0 + std::exp(l_norm));
  return LUFFY_OK;
}

extern "C" int luffy_abi_version(void) { return LUFFY_ABI_VERSION; }

extern "C" const char* luffy_status_string(int status) {
  switch (status) {
    case LUFFY_OK: return "ok";
    case LUFFY_E_INVALID: return "invalid argument";
    case LUFFY_E_UNSUPPORTED: return "unsupported size";
    case LUFFY_E_WORKSPACE: return "workspace too small or misaligned";
    case LUFFY_E_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

extern "C" const char* luffy_last_error(void) { return luffy::g_last_error; }
