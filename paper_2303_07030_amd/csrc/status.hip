// Status strings, thread-local error messages and the version query.
#include <cstdio>

#include "nsd_internal.hpp"

namespace nsd {

namespace {
thread_local char g_msg[512] = "";
}

void set_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
    va_end(ap);
}

void clear_error() { g_msg[0] = '\0'; }

nsd_status fail(nsd_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
    va_end(ap);
    return s;
}

nsd_status check_hip(hipError_t e, const char *what) {
    if (e == hipSuccess) return NSD_OK;
    return fail(NSD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

nsd_status check_launch(const char *what) { return check_hip(hipGetLastError(), what); }

}  // namespace nsd

extern "C" {

const char *nsd_status_string(int status) {
    switch (status) {
        case NSD_OK: return "NSD_OK";
        case NSD_ERR_INVALID_ARG: return "NSD_ERR_INVALID_ARG";
        case NSD_ERR_BAD_FORMAT: return "NSD_ERR_BAD_FORMAT";
        case NSD_ERR_DUPLICATE: return "NSD_ERR_DUPLICATE";
        case NSD_ERR_TOO_LARGE: return "NSD_ERR_TOO_LARGE";
        case NSD_ERR_WORKSPACE: return "NSD_ERR_WORKSPACE";
        case NSD_ERR_UNSUPPORTED: return "NSD_ERR_UNSUPPORTED";
        case NSD_ERR_HIP: return "NSD_ERR_HIP";
        default: return "NSD_ERR_UNKNOWN";
    }
}

const char *nsd_last_error(void) { return nsd::g_msg; }

int nsd_version(void) { return 100; }

}  // extern "C"
