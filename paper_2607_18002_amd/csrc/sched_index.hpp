// Index arithmetic of the persistent tile scheduler (Adaptive Persistent
// Kernel, "Tile-Level Scheduling"; "Tile-aware Latency Model" Eq. (3)): how an
// operation's routed rows become row tiles, weight-sharing groups, per-XCD
// queues and tile numbers.  Pure integer functions, compiled for the device
// (the kernel's instantiation and claims) and for the host (moe_sched_layout,
// which enumerates the same layout so it can be checked on the CPU).
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace moeapk {
namespace sched {

#define MOE_HD __host__ __device__ __forceinline__

// Expert segments are aligned to 32 rows (one MFMA row block).
constexpr int kSegAlign = 32;
constexpr int kXcds = 8;
// Row tiles per op: the group entry holds a row-tile index in 16 bits.
constexpr int kMaxRowTiles = 1 << 16;
// Per-workgroup LDS cache of the own queue's table entries.
constexpr int kTabCache = 64;

// Eq. (3): an expert with m rows runs ceil(m / M_t) row tiles.
MOE_HD int row_tiles(int m, int mt) { return m > 0 ? (m + mt - 1) / mt : 0; }

// Row tile mb (of nt) of an expert with m rows: near-equal heights in whole
// 32-row blocks; tile mb holds blocks [b0, b1) of the segment, so its first
// row is 32*b0 and it has min(m, 32*b1) - 32*b0 valid rows.
// (Products of two row-tile or block counts stay below 2^32: both are below
// kMaxRowTiles = 2^16, so unsigned 32-bit arithmetic is exact; 64-bit
// division is emulated in software on the GPU.)
MOE_HD void tile_rows(int m, int nt, int mb, int& first, int& rows) {
    const uint32_t nb32 = (uint32_t)(m + kSegAlign - 1) / kSegAlign;
    const int b0 = (int)(nb32 * (uint32_t)mb / (uint32_t)nt), b1 = (int)(nb32 * (uint32_t)(mb + 1) / (uint32_t)nt);
    first = b0 * kSegAlign;
    rows = (m < b1 * kSegAlign ? m : b1 * kSegAlign) - first;
}

// Weight-sharing groups: an expert's nt row tiles split into ceil(nt / gmax)
// groups of near-equal size; group j holds row tiles [glo, ghi) of the expert.
MOE_HD int n_groups(int nt, int gmax) { return (nt + gmax - 1) / gmax; }
MOE_HD void group_range(int nt, int ng, int j, int& glo, int& ghi) {
    glo = (int)((uint32_t)nt * (uint32_t)j / (uint32_t)ng);
    ghi = (int)((uint32_t)nt * (uint32_t)(j + 1) / (uint32_t)ng);
}

// The expert whose row tiles include row tile p (scan[e] = first row tile of
// expert e, non-decreasing; p < total): the last e with scan[e] <= p among
// experts that have row tiles.
MOE_HD int expert_of_tile(const int32_t* scan, int E, int total, int p) {
    int lo = 0, hi = E - 1;
    while (lo < hi) {                    // last e with scan[e] <= p
        const int mid = (lo + hi + 1) >> 1;
        if (scan[mid] <= p) lo = mid;
        else hi = mid - 1;
    }
    (void)total;          // an expert with no row tile shares its scan value with the next one, which wins
    return lo;
}

// Queue cut x (1..kXcds-1) of an op with `total` row tiles: the group
// boundary nearest to target = x/kXcds of the row tiles (ties: the lower
// one), so no group spans two queues; cuts are non-decreasing in x.
// scan[e] = first row tile of expert e (exclusive prefix of row_tiles over
// the experts); 0 when no expert has a row tile.  The target lies in the row
// tiles [pos, pos + nt) of one expert, whose group boundaries
// b_j = pos + floor(nt * j / ng) grow with j; with j0 = floor((target - pos) *
// ng / nt), b_j0 <= target <= b_(j0+1), so the nearest boundary is one of the
// two (a boundary of another expert lies at or beyond pos or pos + nt).
MOE_HD int queue_cut(int x, const int32_t* scan, int E, int total, int gmax) {
    if (total <= 0) return 0;
    const int target = (int)((uint32_t)total * (uint32_t)x / kXcds);     // < total
    const int e = expert_of_tile(scan, E, total, target);
    const int pos = scan[e], nt = (e + 1 < E ? scan[e + 1] : total) - pos;
    const int ng = n_groups(nt, gmax);
    const uint32_t j0 = (uint32_t)(target - pos) * (uint32_t)ng / (uint32_t)nt;   // < ng
    const int b0 = pos + (int)((uint32_t)nt * j0 / (uint32_t)ng);
    const int b1 = pos + (int)((uint32_t)nt * (j0 + 1) / (uint32_t)ng);
    return target - b0 <= b1 - target ? b0 : b1;
}

// A row-tile table entry packs everything a claim needs into one 64-bit word:
// bits 0-9 expert, 10-25 row tile within the expert, 26-33 valid rows, 34-63
// first row (capacity * H < 2^31 bounds rows below 2^23).
MOE_HD uint64_t pack_entry(int e, int mb, int rows, int row0) {
    return (uint64_t)((uint32_t)e & 0x3FFu) | ((uint64_t)((uint32_t)mb & 0xFFFFu) << 10) |
           ((uint64_t)((uint32_t)rows & 0xFFu) << 26) | ((uint64_t)(uint32_t)row0 << 34);
}
MOE_HD void unpack_entry(uint64_t ent, int& e, int& mb, int& rows, int& row0) {
    e = (int)(ent & 0x3FFu);
    mb = (int)((ent >> 10) & 0xFFFFu);
    rows = (int)((ent >> 26) & 0xFFu);
    row0 = (int)(ent >> 34);
}
// Group entry of a row tile: first row tile of its group | group size << 16.
MOE_HD uint32_t pack_group(int first, int size) { return (uint32_t)first | ((uint32_t)size << 16); }

// Row tile p of an op (p < total = x_moe): its table and group entries, from
// the experts' counts and segment offsets and scan[e] = first row tile of
// expert e.  Returns false if p does not belong to any expert's tiles (an
// inconsistent count).
MOE_HD bool row_tile_entry(const int32_t* scan, const int32_t* counts, const int32_t* offsets, int E, int total,
                           int mt, int gmax, int p, uint64_t& ent, uint32_t& grp) {
    const int e = expert_of_tile(scan, E, total, p);
    const int c = counts[e], nt = row_tiles(c, mt), pos = scan[e], mb = p - pos;
    if (mb < 0 || mb >= nt) return false;
    const int ng = n_groups(nt, gmax);
    int glo = 0, ghi = nt;
    for (int j = 0; j < ng; ++j) {                   // the near-equal group holding mb
        group_range(nt, ng, j, glo, ghi);
        if (mb < ghi) break;
    }
    int first, rows;
    tile_rows(c, nt, mb, first, rows);
    ent = pack_entry(e, mb, rows, offsets[e] + first);
    grp = pack_group(pos + glo, ghi - glo);
    return true;
}

// Tile t of a queue holding n_mt row tiles starting at m_lo: its stage and
// the row tile p whose group holds it (a group of s row tiles starting at f
// owns the tile numbers [(f - m_lo) * nn, (f - m_lo + s) * nn) of its stage).
MOE_HD void queue_pos(int t, int n_mt, int m_lo, int n1, int n2, int& stage, int& u, int& nn, int& p) {
    const int n1x = n_mt * n1;
    u = t;
    nn = n1;
    stage = 1;
    if (t >= n1x) { stage = 2; u = t - n1x; nn = n2; }
    p = m_lo + u / nn;
}
// ... then, with that group's entry g: column block and row tile (nb < 0: the
// entry is not a valid group of p inside the queue).
MOE_HD void group_tile(uint32_t g, int u, int nn, int m_lo, int n_mt, int p, int& mtile, int& nb) {
    const int f = (int)(g & 0xFFFFu), sz = (int)(g >> 16);
    if (sz < 1 || f < m_lo || p < f || p >= f + sz || f + sz > m_lo + n_mt) { nb = -1; mtile = -1; return; }
    const int w = u - (f - m_lo) * nn;
    nb = w / sz;
    mtile = f + (w - nb * sz);
}

// Slot of row tile p in a workgroup's LDS cache of its own queue's entries
// (the queue's range starts at lo; cnt entries were filled, at most
// kTabCache), or -1 when p is not cached.
MOE_HD int cache_slot(int p, int lo, int cnt) {
    return (lo >= 0 && cnt <= kTabCache && p >= lo && p < lo + cnt) ? p - lo : -1;
}

#undef MOE_HD

}  // namespace sched
}  // namespace moeapk
