// Status strings, thread-local error messages and the version query.
#include <cstdio>
#include <vector>

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

namespace {
struct Probe {
    int id = 0;
    std::vector<hipEvent_t> start, stop;
    int32_t count = 0;
};
thread_local Probe g_probe;
}  // namespace

void probe_begin(int kernel_id, hipStream_t st) {
    if (g_probe.id != kernel_id || g_probe.start.empty()) return;
    (void)hipEventRecord(g_probe.start[g_probe.count % g_probe.start.size()], st);
}

void probe_end(int kernel_id, hipStream_t st) {
    if (g_probe.id != kernel_id || g_probe.stop.empty()) return;
    (void)hipEventRecord(g_probe.stop[g_probe.count % g_probe.stop.size()], st);
    ++g_probe.count;
}

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

nsd_status nsd_probe_set(int kernel_id, void *const *start_events, void *const *stop_events,
                         int32_t n) {
    NSD_REQUIRE(kernel_id > 0 && kernel_id <= NSD_KERNEL_BATAX_ROWS, "unknown kernel id %d", kernel_id);
    NSD_REQUIRE(n >= 1 && start_events && stop_events, "need n >= 1 event pairs");
    nsd::Probe p;
    p.id = kernel_id;
    for (int32_t i = 0; i < n; ++i) {
        NSD_REQUIRE(start_events[i] && stop_events[i], "event %d is NULL", i);
        p.start.push_back(static_cast<hipEvent_t>(start_events[i]));
        p.stop.push_back(static_cast<hipEvent_t>(stop_events[i]));
    }
    nsd::g_probe = p;
    return NSD_OK;
}

nsd_status nsd_probe_count(int32_t *count) {
    NSD_REQUIRE(count != nullptr, "count is NULL");
    *count = nsd::g_probe.count;
    return NSD_OK;
}

nsd_status nsd_probe_clear(void) {
    nsd::g_probe = nsd::Probe{};
    return NSD_OK;
}

}  // extern "C"
