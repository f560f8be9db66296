// Status strings, thread-local error text, device queries.
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "common.hpp"

namespace bandlu {

static thread_local char g_last_error[512];

void clear_error() { g_last_error[0] = '\0'; }

void set_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
}

int hip_fail(hipError_t e, const char *what) {
    set_error("%s: %s", what, hipGetErrorString(e));
    return BANDLU_ERR_HIP;
}

int device_cu_count() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return 256;
    return cus;
}

}  // namespace bandlu

extern "C" const char *band_status_string(int status) {
    if (status == BANDLU_OK) return "ok";
    if (status == BANDLU_ERR_HIP) return "HIP runtime or launch failure";
    if (status == BANDLU_ERR_UNSUPPORTED) return "unsupported argument combination";
    if (status < 0 && status > -100) return "invalid argument";
    return "unknown status";
}

extern "C" const char *band_last_error(void) { return bandlu::g_last_error; }
