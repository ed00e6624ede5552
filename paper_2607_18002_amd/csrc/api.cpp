// Host-side plumbing of the C ABI: error strings, thread-local last error,
// device checks and the pure host helpers of Eq. (3) and Eq. (4).
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "common.hpp"

namespace {
thread_local char g_last_error[512] = "";

struct DevInfo {
    bool probed = false;
    bool ok = false;
    int cu = 0;
    int wallclock_khz = 0;
};
constexpr int kMaxDevices = 64;
DevInfo g_dev[kMaxDevices];
std::mutex g_dev_mu;
}  // namespace

namespace moeapk_host {

moe_status_t fail(moe_status_t code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return code;
}

moe_status_t check_device(int* cu_count, int* wallclock_khz) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return fail(MOE_ERR_HIP, "hipGetDevice failed");
    if (dev < 0 || dev >= kMaxDevices) return fail(MOE_ERR_UNSUPPORTED, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_dev_mu);
    DevInfo& d = g_dev[dev];
    if (!d.probed) {
        hipDeviceProp_t p;
        if (hipGetDeviceProperties(&p, dev) != hipSuccess) return fail(MOE_ERR_HIP, "hipGetDeviceProperties failed");
        d.ok = std::strncmp(p.gcnArchName, "gfx950", 6) == 0;
        d.cu = p.multiProcessorCount;
        int wc = 0;
        if (hipDeviceGetAttribute(&wc, hipDeviceAttributeWallClockRate, dev) != hipSuccess) wc = 100000;
        d.wallclock_khz = wc > 0 ? wc : 100000;
        d.probed = true;
        if (!d.ok) {
            return fail(MOE_ERR_UNSUPPORTED, "device %d is %s; this library is built for gfx950 only", dev,
                        p.gcnArchName);
        }
    }
    if (!d.ok) return fail(MOE_ERR_UNSUPPORTED, "device %d is not gfx950", dev);
    if (cu_count) *cu_count = d.cu;
    if (wallclock_khz) *wallclock_khz = d.wallclock_khz;
    return MOE_OK;
}

}  // namespace moeapk_host

extern "C" {

const char* moe_status_string(moe_status_t s) {
    switch (s) {
        case MOE_OK: return "MOE_OK";
        case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
        case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
        case MOE_ERR_CAPACITY: return "MOE_ERR_CAPACITY";
        case MOE_ERR_HIP: return "MOE_ERR_HIP";
        case MOE_ERR_ABORTED: return "MOE_ERR_ABORTED";
        case MOE_ERR_TIMEOUT: return "MOE_ERR_TIMEOUT";
        case MOE_ERR_BAD_EXPERT: return "MOE_ERR_BAD_EXPERT";
        case MOE_ERR_INTERNAL: return "MOE_ERR_INTERNAL";
        default: return "MOE_ERR_UNKNOWN";
    }
}

const char* moe_last_error(void) { return g_last_error; }

size_t moe_abi_sizeof(int32_t which) {
    switch (which) {
        case 0: return sizeof(moe_op_desc);
        case 1: return sizeof(moe_sched_config);
        case 2: return sizeof(moe_trace_rec);
        case 3: return sizeof(moe_op_stats);
        case 4: return sizeof(moe_route_args);
        case 5: return sizeof(moe_permute_args);
        case 6: return sizeof(moe_combine_args);
        default: return 0;
    }
}

int32_t moe_x_moe(const int32_t* counts_host, int32_t E_local, int32_t M_t) {
    if (!counts_host || E_local < 0 || M_t <= 0) return -1;
    int64_t s = 0;
    for (int32_t e = 0; e < E_local; ++e)
        if (counts_host[e] > 0) s += moeapk::ceil_div(counts_host[e], M_t);
    return (int32_t)s;
}

int32_t moe_decode_quota(int32_t q, int32_t x_moe, int32_t x_moe_expected, int32_t q_max, int32_t c) {
    return moeapk::decode_quota(q, x_moe, x_moe_expected, q_max, c);
}

}  // extern "C"
