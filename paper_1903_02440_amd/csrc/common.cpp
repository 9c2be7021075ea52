// Error state and version of libspyke.
#include <cstdio>
#include <string>

#include "common.hpp"

namespace spk {

static thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int ok() {
    g_last_error.clear();
    return SPK_OK;
}

int check_launch(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(SPK_E_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

}  // namespace spk

extern "C" int spk_version(void) { return (0 << 16) | (1 << 8) | 0; }

extern "C" const char *spk_last_error(void) { return spk::g_last_error.c_str(); }
