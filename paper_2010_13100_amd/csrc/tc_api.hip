// Status codes, per-thread error messages and launch checks of libtc.
#include <cstdarg>
#include <cstring>

#include "tc_internal.h"

namespace tc {
namespace {
thread_local char g_error[512] = "";
}

void set_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof(g_error), fmt, ap);
    va_end(ap);
}

void clear_error() { g_error[0] = '\0'; }

int device_cus() {
    constexpr int kMaxDevices = 64;
    static int cached[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
    if (dev < kMaxDevices) {
        const int c = __atomic_load_n(&cached[dev], __ATOMIC_RELAXED);
        if (c > 0) return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        return 256;
    if (dev < kMaxDevices) __atomic_store_n(&cached[dev], cus, __ATOMIC_RELAXED);
    return cus;
}

tc_status check_launch(const char *what) {
    const hipError_t e = hipGetLastError();
    if (e == hipSuccess) return TC_OK;
    set_error("%s: %s", what, hipGetErrorString(e));
    return TC_ERR_HIP;
}

}  // namespace tc

extern "C" const char *tc_status_string(tc_status status) {
    // callers may pass any int; read it as one (an enum load of a value
    // outside the enumerators' range would be undefined in C++)
    int32_t code = 0;
    std::memcpy(&code, &status, sizeof(code));
    switch (code) {
        case TC_OK: return "TC_OK";
        case TC_ERR_INVALID_ARG: return "TC_ERR_INVALID_ARG";
        case TC_ERR_UNSUPPORTED: return "TC_ERR_UNSUPPORTED";
        case TC_ERR_WORKSPACE: return "TC_ERR_WORKSPACE";
        case TC_ERR_HIP: return "TC_ERR_HIP";
    }
    return "TC_ERR_UNKNOWN";
}

extern "C" const char *tc_last_error(void) { return tc::g_error; }

extern "C" int32_t tc_abi_version(void) { return TC_ABI_VERSION; }
