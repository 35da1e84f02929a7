// Status codes, per-thread error messages and pinned mapped host memory.
#include <string>

#include "internal.hpp"

namespace {
thread_local std::string g_last_error;
thread_local ss::kernel_timing g_timing;
}

namespace ss {

ss_status fail(ss_status code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

void clear_error() { g_last_error.clear(); }

kernel_timing take_kernel_timing()
{
    kernel_timing t = g_timing;
    g_timing = kernel_timing{};
    return t;
}

void set_kernel_timing(hipEvent_t start, hipEvent_t stop) { g_timing = kernel_timing{start, stop}; }

ss_status check_launch(const char *what)
{
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(SS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return SS_OK;
}

}  // namespace ss

extern "C" {

int ss_abi_version(void) { return SS_ABI_VERSION; }

const char *ss_status_string(ss_status s)
{
    switch (s) {
    case SS_OK: return "ok";
    case SS_ERR_INVALID_ARG: return "invalid argument";
    case SS_ERR_UNSUPPORTED: return "unsupported shape or parameter";
    case SS_ERR_CAPACITY: return "selection exceeds cache capacity";
    case SS_ERR_OOM: return "out of memory or buffer too small";
    case SS_ERR_HIP: return "HIP runtime error";
    case SS_ERR_TIMEOUT: return "timed out waiting for the GPU";
    default: return "unknown status";
    }
}

const char *ss_last_error(void) { return g_last_error.c_str(); }

ss_status ss_host_alloc_mapped(size_t bytes, unsigned flags, void **host_ptr, void **dev_ptr)
{
    SS_CHECK_ARG(host_ptr && dev_ptr, "ss_host_alloc_mapped: null output pointer");
    SS_CHECK_ARG(flags <= 1, "ss_host_alloc_mapped: flags must be 0 or 1");
    *host_ptr = nullptr;
    *dev_ptr = nullptr;
    if (bytes == 0) return SS_OK;
    unsigned hf = hipHostMallocMapped | (flags == 1 ? hipHostMallocNonCoherent : hipHostMallocCoherent);
    void *h = nullptr;
    hipError_t e = hipHostMalloc(&h, bytes, hf);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return ss::fail(SS_ERR_OOM, "hipHostMalloc(%zu bytes): %s", bytes, hipGetErrorString(e));
    }
    void *d = nullptr;
    e = hipHostGetDevicePointer(&d, h, 0);
    if (e != hipSuccess) {
        (void)hipHostFree(h);
        return ss::fail(SS_ERR_HIP, "hipHostGetDevicePointer: %s", hipGetErrorString(e));
    }
    *host_ptr = h;
    *dev_ptr = d;
    ss::clear_error();
    return SS_OK;
}

ss_status ss_time_next_kernel(void *start_event, void *stop_event)
{
    ss::set_kernel_timing(reinterpret_cast<hipEvent_t>(start_event), reinterpret_cast<hipEvent_t>(stop_event));
    return SS_OK;
}

ss_status ss_host_free(void *host_ptr)
{
    if (!host_ptr) return SS_OK;
    hipError_t e = hipHostFree(host_ptr);
    if (e != hipSuccess) return ss::fail(SS_ERR_HIP, "hipHostFree: %s", hipGetErrorString(e));
    return SS_OK;
}

}  // extern "C"
