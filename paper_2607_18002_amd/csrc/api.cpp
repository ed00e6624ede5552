// Host-side plumbing of the C ABI: error strings, thread-local last error,
// device checks and the pure host helpers of Eq. (3) and Eq. (4).
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include <vector>

#include "common.hpp"
#include "sched_index.hpp"

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

int32_t moe_sched_layout(const int32_t* counts, const int32_t* offsets, int32_t E_local, int32_t M_t, int32_t gmax,
                         int32_t n1, int32_t n2, int32_t max_row_tiles, int32_t* row_tiles, int32_t* groups,
                         int32_t* queues, int64_t max_tiles, int32_t* tiles) {
    namespace S = moeapk::sched;
    if (!counts || !offsets || E_local < 1 || M_t < 1 || gmax < 1 || n1 < 1 || n2 < 1 || max_row_tiles < 0)
        return -1;
    std::vector<int32_t> scan(E_local);
    int total = 0;
    for (int e = 0; e < E_local; ++e) {
        if (counts[e] < 0) return -1;
        scan[e] = total;
        total += S::row_tiles(counts[e], M_t);
    }
    if (total > max_row_tiles || total >= S::kMaxRowTiles || (int64_t)total * (n1 + n2) > max_tiles) return -1;
    // the instantiation: table and group entries of every row tile
    std::vector<uint64_t> table(total > 0 ? total : 1);
    std::vector<uint32_t> grp(total > 0 ? total : 1);
    for (int p = 0; p < total; ++p)
        if (!S::row_tile_entry(scan.data(), counts, offsets, E_local, total, M_t, gmax, p, table[p], grp[p])) return -2;
    for (int p = 0; p < total; ++p) {
        int e, mb, rows, row0;
        S::unpack_entry(table[p], e, mb, rows, row0);
        row_tiles[4 * p] = e;
        row_tiles[4 * p + 1] = mb;
        row_tiles[4 * p + 2] = rows;
        row_tiles[4 * p + 3] = row0;
        groups[2 * p] = (int32_t)(grp[p] & 0xFFFFu);
        groups[2 * p + 1] = (int32_t)(grp[p] >> 16);
    }
    int cut[S::kXcds + 1];
    cut[0] = 0;
    cut[S::kXcds] = total;
    for (int x = 1; x < S::kXcds; ++x) cut[x] = S::queue_cut(x, scan.data(), E_local, total, gmax);
    for (int x = 0; x < S::kXcds; ++x) {
        queues[2 * x] = cut[x];
        queues[2 * x + 1] = cut[x + 1] - cut[x];
    }
    // every claim of every queue, resolved as a workgroup of each XCD would
    // resolve it (its LDS cache holds its own queue's entries when they fit);
    // all eight must agree, as a claimed tile may be taken by any of them
    int64_t n = 0;
    for (int x = 0; x < S::kXcds; ++x) {
        const int m_lo = cut[x], n_mt = cut[x + 1] - cut[x];
        for (int t = 0; t < n_mt * (n1 + n2); ++t) {
            int stage = 0, ref_mtile = -2, ref_nb = -2;
            for (int y = 0; y < S::kXcds; ++y) {
                // workgroup of XCD y: its cache holds its own queue's first cnt
                // entries when cnt fits, and unfilled slots hold garbage
                const int lo = cut[y], cnt = cut[y + 1] - cut[y];
                uint32_t cache_g[S::kTabCache];
                uint64_t cache_e[S::kTabCache];
                for (int i = 0; i < S::kTabCache; ++i) {
                    const bool filled = cnt <= S::kTabCache && i < cnt;
                    cache_g[i] = filled ? grp[lo + i] : 0xA5A5A5A5u;
                    cache_e[i] = filled ? table[lo + i] : 0xA5A5A5A5A5A5A5A5ull;
                }
                int st, u, nn, p, mtile, nb;
                S::queue_pos(t, n_mt, m_lo, n1, n2, st, u, nn, p);
                const int cg = S::cache_slot(p, lo, cnt);
                if (cg >= S::kTabCache) return -2;
                const uint32_t g = cg >= 0 ? cache_g[cg] : (p >= 0 && p < total ? grp[p] : 0u);
                S::group_tile(g, u, nn, m_lo, n_mt, p, mtile, nb);
                if (y == 0) { stage = st; ref_mtile = mtile; ref_nb = nb; }
                else if (mtile != ref_mtile || nb != ref_nb) return -2;
                const int ce = S::cache_slot(mtile, lo, cnt);
                if (ce >= S::kTabCache) return -2;
                const uint64_t ent = ce >= 0 ? cache_e[ce] : (mtile >= 0 && mtile < total ? table[mtile] : 0ull);
                if (mtile < 0 || ent != table[mtile]) return -2;
            }
            tiles[4 * n] = x;
            tiles[4 * n + 1] = stage;
            tiles[4 * n + 2] = ref_mtile;
            tiles[4 * n + 3] = ref_nb;
            ++n;
        }
    }
    return total;
}

}  // extern "C"
