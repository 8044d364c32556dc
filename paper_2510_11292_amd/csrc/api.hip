// Status strings, the thread-local last-error text, and the local-window rule.
#include <stdarg.h>

#include <mutex>
#include <unordered_map>

#include "common.h"

namespace louiskv {
namespace {
thread_local char g_err[1024] = "";
}
const char* g_err_text() { return g_err; }

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return status;
}

int device_view_of_host_pool(const void* p, void** dev) {
  if (!p) {
    *dev = nullptr;
    return LOUISKV_OK;
  }
  hipPointerAttribute_t attr;
  const hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess || attr.type != hipMemoryTypeHost || attr.devicePointer == nullptr) {
    (void)hipGetLastError();   // clear the lookup's error so that later calls do not report it
    return fail(LOUISKV_ERR_UNSUPPORTED,
                "pool_on_host=1 needs pinned, device-mapped host memory (hipHostMalloc); %p is not", p);
  }
  *dev = attr.devicePointer;
  return LOUISKV_OK;
}

namespace {
std::mutex g_lds_mu;
std::unordered_map<const void*, size_t> g_static_lds;   // per kernel
int g_max_lds[64] = {};                                  // per device
int g_cus[64] = {};                                      // per device
}  // namespace

int device_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lock(g_lds_mu);
  if (!g_cus[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    g_cus[dev] = n;
  }
  return g_cus[dev];
}

int check_lds(const void* kernel, size_t dynamic_lds) {
  int dev = 0;
  LKV_CHECK_HIP(hipGetDevice(&dev));
  size_t stat = 0;
  int limit = 0;
  {
    std::lock_guard<std::mutex> lock(g_lds_mu);
    auto it = g_static_lds.find(kernel);
    if (it == g_static_lds.end()) {
      hipFuncAttributes attr;
      LKV_CHECK_HIP(hipFuncGetAttributes(&attr, kernel));
      it = g_static_lds.emplace(kernel, attr.sharedSizeBytes).first;
    }
    stat = it->second;
    if (dev >= 0 && dev < 64) {
      if (!g_max_lds[dev]) {
        int a = 0, b = 0;
        LKV_CHECK_HIP(hipDeviceGetAttribute(&a, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
        LKV_CHECK_HIP(hipDeviceGetAttribute(&b, hipDeviceAttributeSharedMemPerBlockOptin, dev));
        g_max_lds[dev] = std::max(a, b);
      }
      limit = g_max_lds[dev];
    }
  }
  if (limit <= 0 || stat + dynamic_lds > (size_t)limit)
    return fail(LOUISKV_ERR_UNSUPPORTED, "launch needs %zu bytes of LDS (%zu static + %zu dynamic), the device has %d",
                stat + dynamic_lds, stat, dynamic_lds, limit);
  return LOUISKV_OK;
}

}  // namespace louiskv

extern "C" int louiskv_abi_version(void) { return LOUISKV_ABI_VERSION; }

extern "C" const char* louiskv_status_str(int status) {
  switch (status) {
    case LOUISKV_OK: return "ok";
    case LOUISKV_ERR_NULL: return "required pointer is NULL";
    case LOUISKV_ERR_SHAPE: return "inconsistent or out-of-range sizes";
    case LOUISKV_ERR_DTYPE: return "unknown dtype";
    case LOUISKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case LOUISKV_ERR_WORKSPACE: return "workspace missing or too small";
    case LOUISKV_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

extern "C" const char* louiskv_last_error(void) { return louiskv::g_err_text(); }

extern "C" int louiskv_window_info(int32_t step, int32_t window, int32_t seg_len, int32_t* evicted_segment,
                                   int32_t* n_evicted, int32_t* n_local, int32_t* local_start) {
  if (step < 0 || seg_len < 1 || window < seg_len || window % seg_len != 0)
    return louiskv::fail(LOUISKV_ERR_SHAPE, "window=%d must be a positive multiple of seg_len=%d, step=%d >= 0",
                         window, seg_len, step);
  const int32_t ev = step >= window && (step - window) % seg_len == 0 ? (step - window) / seg_len : -1;
  const int32_t nev = step >= window ? (step - window) / seg_len + 1 : 0;
  const int64_t first_live = (int64_t)nev * seg_len;
  if (evicted_segment) *evicted_segment = ev;
  if (n_evicted) *n_evicted = nev;
  if (n_local) *n_local = (int32_t)(step + 1 - first_live);
  if (local_start) *local_start = (int32_t)(first_live % window);
  return LOUISKV_OK;
}
