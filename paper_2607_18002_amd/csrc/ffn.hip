// a3-a6: the SwiGLU expert FFN as one adaptive persistent kernel.
//
// Paper passages: Adaptive Persistent Kernel -- "Tile-Level Scheduling" (a
// tile is the scheduling unit; phases switch only when a tile commits;
// operation templates are instantiated into a decode or a prefill queue when
// their ready signal is seen), "Bounded Tile-level Preemption" (a decision is
// read once per tile boundary and broadcast to the whole cooperating unit),
// "Online SM Reallocation" Eq. (4) (decode quota under contention, a lone
// phase takes everything), "Tile-aware Latency Model" Eq. (3) (the number of
// executed row tiles); Evaluation "Implementation" (two grouped GEMMs and the
// activation fused into one long-lived kernel).
//
// MI355X design.  One 256-thread workgroup per CU, fixed grid.  CDNA4 has no
// thread-block clusters, so the scheduling unit is the workgroup: at every
// tile boundary wave 0 commits the finished tile, polls the operation words
// (one lane per operation), claims the next tile with one device-scope atomic
// and broadcasts it through LDS; the whole workgroup runs the tile.  A
// template whose inputs were in place at the launch is built ahead of its
// ready signal (row tiles, queues, counters) by a workgroup that never
// prefers decode; the signal then only flips its state word, and the
// workgroup that flips it claims the first tile in the same boundary.  Each
// operation's tiles are numbered GEMM-1 tiles first (row-tile major), then
// GEMM-2 tiles; a GEMM-2 tile waits (bounded) on a per-row-tile counter that
// GEMM-1 tiles bump once their h rows are visible.  Every claimed tile belongs
// to a running workgroup, so the dependency waits cannot deadlock.  Commits
// are counted with atomics whose result nobody waits for; an operation whose
// polled count of committed tiles reached its total is finished by the
// workgroup that wins its ACTIVE -> FINISHING transition.  An op with a fused
// combine turns COMBINING once its GEMM tiles have all committed; its combine
// tiles (weighted sums of y_perm rows back into token order) are then claimed
// from one shared counter, and it finishes after the last of them.
//
// Coherence across the eight XCD-private L2 caches.  An agent-scope acquire
// invalidates the whole L2 of the XCD, which would destroy weight reuse if it
// sat on the polling path.  So every scheduler word is read with relaxed
// device-scope atomics (coherent loads that invalidate nothing).  Tile outputs
// (h, y_perm) are written with device-coherent stores (sc1) that reach the
// coherence point by themselves, and every wave waits for its own stores
// before the workgroup barrier that precedes the commit, so bumping a counter
// needs no L2 write-back of its own.  Consumers of h never invalidate: within
// one launch a workgroup reads an h row only after the row's GEMM-1 tiles
// committed and never before, so no L1/L2 can hold a stale copy of it (launch
// boundaries make earlier launches' copies coherent).  Row-tile tables, which
// are written with ordinary stores, are published with a release by every
// wave that wrote them.  The one acquire per operation is taken by the
// workgroup that finishes it, before it publishes the done word.
#include <cstring>
#include <mutex>

#include "sched_index.hpp"
#include "tile_bf16.hpp"
#include "tile_bf16_tall.hpp"
#include "tile_fp8.hpp"

namespace {

using namespace moeapk;
using sched::kMaxRowTiles;
using sched::kSegAlign;
using sched::kTabCache;
using sched::kXcds;

using ShapeP = TileShape<192, 256, 64>;    // bf16 prefill: 192 x 256 tall tile, K step 64
using ShapeD = TileShape<128, 256, 64>;    // bf16 decode : 128 x 256 tile, K step 64
// bf16 decode beside prefill ops: the same tile with its weights loaded
// non-temporal.  A decode op's weight slice serves its one or two row tiles
// and is then dead in the L2, where it would evict the slices and activation
// rows that a prefill group still shares (4 layers of 8192 prefill + 1024
// decode tokens: +1.3%).  Decode alone gains nothing from it, so launches
// without prefill ops keep the plain loads.
using ShapeDS = TileShape<128, 256, 64, kLoadStream>;
using ShapeF8 = TileShapeF8<128, 256>;     // fp8 (both phases): 128 x 256 tile, K step 128 (one scale block)
using ShapeF8S = TileShapeF8<128, 256, kLoadStream>;   // fp8 decode beside prefill ops (as ShapeDS)
constexpr int kMax2(int a, int b) { return a > b ? a : b; }
constexpr int kLdsBytes = kMax2(kMax2(TallLds<ShapeP>::bytes, ShapeD::LDS), ShapeF8::LDS);
// Expert segments are aligned to 32 rows (one MFMA row block).  An expert's m
// rows are cut into ceil(m / M_t) row tiles of near-equal height in whole
// 32-row blocks (M_t = the class's tallest tile), so the row tiles that share
// a weight slice run about equally long and stay in step (sched_index.hpp).

enum : int32_t { CLS_P_BF16 = 0, CLS_D_BF16 = 1, CLS_FP8 = 2, CLS_D_BF16_S = 3, CLS_FP8_S = 4 };
__host__ __device__ __forceinline__ bool is_fp8_cls(int cls) { return cls == CLS_FP8 || cls == CLS_FP8_S; }
enum : int32_t { ST_WAIT = 0, ST_INIT = 1, ST_ACTIVE = 2, ST_DONE = 3, ST_FINISHING = 4, ST_COMBINING = 5 };
// A template built ahead of its ready signal (row tiles, queues and counters
// in place, nothing claimable) waits in a state word that also carries what
// its activation needs: ST_BUILT | (no row tiles) << 4 | q' << 5.
constexpr int32_t ST_BUILT = 6;
__device__ __forceinline__ bool is_built(int32_t s) { return (s & 15) == ST_BUILT; }
__device__ __forceinline__ int32_t built_word(int xm, int qd) { return ST_BUILT | (xm == 0 ? 16 : 0) | (qd << 5); }
constexpr int kCombTokens = 32;           // tokens per fused-combine tile
enum : int32_t { CMD_EXIT = 0, CMD_TILE = 1, CMD_INST = 2, CMD_IDLE = 3 };

struct OpArg {
    const int32_t* counts;
    const int32_t* offsets;
    const uint16_t* x;         // bf16 elements, or fp8 codes (bytes) for the fp8 classes: x_perm, or x when gathered
    const uint16_t* wgu;
    const uint16_t* wd;
    uint16_t* h;
    uint16_t* y;
    const float* xs;           // fp8 scales: x_perm, gate/up weights, down weights, h
    const float* wgus;
    const float* wds;
    float* hs;
    uint32_t* done_word;
    const int32_t* rmap;       // gathered GEMM-1 operand: row -> assignment (x row = assignment / top_k), else NULL
    const int32_t* a2r;        // fused combine: assignment -> row, topk weights, output (y NULL: none)
    const float* tw;
    void* yc;
    int32_t cls, phase, layer, E, H, I, capacity, mt, n1, n2, max_mtiles, table_off, g1_off, grp_off, T, top_k;
    int32_t ct, ck, y_f32, n3;  // combine: tokens, slots per token, fp32 output, combine tiles
    int32_t rel, qtab_off;      // rel: the op has a release word; qtab_off: per-queue copies of table entries
};

struct KArgs {
    OpArg op[MOE_MAX_OPS];
    int32_t n_ops, q, q_max, x_star, c, gmax;
    int32_t pre_wg;            // prefill tiles are claimed ahead only by workgroups >= pre_wg
    int32_t pre_dec_all;       // no prefill op in the launch: every workgroup claims decode tiles ahead
    int32_t split;             // static partition: decode only below pre_wg, prefill only at or above
    int32_t inst_wg;           // decode templates are instantiated by workgroups below this (0: any)
    int64_t spin_limit;
    const uint32_t* abort_word;
    moe_trace_rec* trace;
    int64_t trace_per_wg;      // records per workgroup block (trace: n_wg blocks of this many)
    moe_op_stats* stats;
    int32_t* status;
    char* ws;
};

// Run-time state of an op: every access is an atomic (one L2 line per op).
// left: -(tiles not yet committed) once the op is instantiated, counting up to
// 0 with one increment per commit; INT_MIN before, so a stale read is never 0.
// With a fused combine the count holds the GEMM tiles and the n3 combine tiles:
// it passes -n3 when the last GEMM tile commits (ACTIVE -> COMBINING) and 0
// when the last combine tile does.  cclaim: the combine tiles' claim counter.
struct OpDyn {
    int32_t state, cclaim, left, x_moe;
    int32_t total, pad_b, quota, pad0;
    unsigned long long t_ready, t_first, t_done, t_seen;
    char pad[128 - 64];
};
static_assert(sizeof(OpDyn) == 128, "one L2 line per op");

// Readiness fields of an op: written by the init kernel, read-only during the launch.
struct OpStatic {
    int32_t phase, dep, pad0, pad1;
    const uint32_t* rel_word;
    int64_t rel_after, gap;                    // ticks; rel_after < 0: no time condition
    char pad[128 - 40];
};
static_assert(sizeof(OpStatic) == 128, "one L2 line per op");

struct Hdr {
    unsigned long long t0;                   // first workgroup's entry (wall-clock ticks)
    int32_t ops_done, quota, n_wg, stop;     // n_wg: the launch's workgroups (the trace's block count)
    unsigned long long t_init, t_exit;       // init kernel done; last workgroup's exit
};

// One tile queue per (op, XCD): the op's row tiles are cut into kXcds
// contiguous ranges [m_lo, m_lo + n_mt), balanced by row tiles and cut only
// between groups (below); queue x holds the GEMM-1 tiles of its range, then
// its GEMM-2 tiles.  Workgroups claim from their own XCD's queue, so the
// activation rows and h of a row tile and the weight slices of a group stay
// in one L2; a workgroup whose queue is empty steals from the others.  claim
// is an atomic counter; size / m_lo / n_mt are written once at instantiation.
struct XQueue {
    int32_t claim, size, m_lo, n_mt;
    char pad[128 - 16];
};
static_assert(sizeof(XQueue) == 128, "one L2 line per queue");

// Groups: an expert's row tiles are split into ceil(n / gmax) groups of
// near-equal size (gmax = group_row_tiles), and a queue runs each group column
// block by column block, the group's row tiles back to back, so one fetch of
// a weight slice into the XCD's L2 serves every row tile of the group while
// it is hot.  A group never holds two experts, so an expert's weights are
// streamed once per group.  grp[p] = first row tile | size << 16 of the group
// holding row tile p.
constexpr int kDefaultGroup = 8;
constexpr int kMaxGroup = 64;

constexpr size_t kHdrBytes = 256;
constexpr size_t kDynOff = kHdrBytes;
constexpr size_t kStaticOff = kDynOff + MOE_MAX_OPS * sizeof(OpDyn);
constexpr size_t kXqOff = kStaticOff + MOE_MAX_OPS * sizeof(OpStatic);
constexpr size_t kArraysOff = kXqOff + MOE_MAX_OPS * kXcds * sizeof(XQueue);

__device__ __forceinline__ Hdr* hdr_of(char* ws) { return (Hdr*)ws; }
__device__ __forceinline__ OpDyn* dyn_of(char* ws) { return (OpDyn*)(ws + kDynOff); }
__device__ __forceinline__ OpStatic* static_of(char* ws) { return (OpStatic*)(ws + kStaticOff); }
__device__ __forceinline__ char* arr_of(char* ws) { return ws + kArraysOff; }
__device__ __forceinline__ XQueue* xq_of(char* ws, int o, int x) { return (XQueue*)(ws + kXqOff) + o * kXcds + x; }

// ----------------------------------------------------------------------------- init
struct InitArgs {
    const uint32_t* rel_words[MOE_MAX_OPS];
    int64_t rel_after[MOE_MAX_OPS];
    int64_t gaps[MOE_MAX_OPS];
    int32_t deps[MOE_MAX_OPS];
    int32_t phases[MOE_MAX_OPS];
    int32_t n_ops, ws_vec;           // ws_vec: 16-byte words of scheduler state
    char* ws;
    int32_t* status;
};

// Zeroes the scheduler state (16-byte stores; the row-tile tables too, so an
// entry read before it was written reads as invalid rather than as a previous
// launch's tile) and writes the readiness fields; launched on the same stream
// right before the persistent kernel.  Workgroup 0 zeroes the header, op and
// queue lines and then writes the fields; the others zero the per-op arrays.
__global__ __launch_bounds__(256) void apk_init_kernel(const InitArgs a) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    const int head = (int)(kArraysOff / 16);
    if (blockIdx.x > 0) {
        for (int i = head + (blockIdx.x - 1) * 256 + threadIdx.x; i < a.ws_vec; i += (gridDim.x - 1) * 256)
            ((u32x4*)a.ws)[i] = z;
        return;
    }
    for (int i = threadIdx.x; i < head && i < a.ws_vec; i += 256) ((u32x4*)a.ws)[i] = z;
    __syncthreads();
    if (threadIdx.x == 0) {
        OpStatic* st = static_of(a.ws);
        for (int o = 0; o < a.n_ops; ++o) {
            st[o].phase = a.phases[o];
            st[o].dep = a.deps[o];
            st[o].rel_word = a.rel_words[o];
            st[o].rel_after = a.rel_after[o];
            st[o].gap = a.gaps[o];
            dyn_of(a.ws)[o].left = INT32_MIN;
        }
        *a.status = MOE_OK;
        hdr_of(a.ws)->t_init = wall_ticks();
    }
}

// ----------------------------------------------------------------------------- tiles
// bf16 tiles: TALL selects the 192-row prefill tile (tile_bf16_tall.hpp),
// else the 128-row tile (tile_bf16.hpp); both take the same operands.
template <class S, bool TALL, class Hook>
__device__ __forceinline__ void run_tile_cls(const OpArg& op, int stage, int row0, int rows32, int nb, int e, char* lds,
                                             Hook hook) {
    const long H = op.H, I = op.I;
    if (stage == 1) {
        const bool g = op.rmap != nullptr;
        const uint16_t* A = g ? op.x : op.x + row0 * H;
        const uint16_t* B = op.wgu + (long)e * 2 * I * H + (long)nb * (S::BN / 2) * H;
        uint16_t* out = op.h + row0 * I + nb * (S::BN / 2);
        const int32_t* rmap = g ? op.rmap + row0 : nullptr;
        if constexpr (TALL)
            gemm_tile_tall_rows<S, true>(rows32, A, (int)H, B, (int)H, (int)I, (int)H, out, (int)I, lds, rmap,
                                         op.top_k, op.T, hook);
        else
            gemm_tile_bf16_rows<S, true, true>(rows32, A, (int)H, B, (int)H, (int)I, (int)H, out, (int)I, lds, rmap,
                                               op.top_k, op.T, hook);
    } else {
        const uint16_t* A = op.h + row0 * I;
        const uint16_t* B = op.wd + (long)e * H * I + (long)nb * S::BN * I;
        uint16_t* out = op.y + row0 * H + nb * S::BN;
        if constexpr (TALL)
            gemm_tile_tall_rows<S, false>(rows32, A, (int)I, B, (int)I, 0, (int)I, out, (int)H, lds, nullptr, 1, 0,
                                          hook);
        else
            gemm_tile_bf16_rows<S, false, true>(rows32, A, (int)I, B, (int)I, 0, (int)I, out, (int)H, lds, nullptr, 1,
                                                0, hook);
    }
}

// fp8: GEMM-1 tiles cover 128 h columns (one h scale group), GEMM-2 tiles 256 y columns.
template <class S, class Hook>
__device__ __forceinline__ void run_tile_fp8(const OpArg& op, int stage, int row0, int rows32, int nb, int e,
                                             char* lds, Hook hook) {
    const long H = op.H, I = op.I;
    const uint8_t* x = (const uint8_t*)op.x;
    uint8_t* h = (uint8_t*)op.h;
    if (stage == 1) {
        const int n0 = nb * (S::BN / 2);
        const bool g = op.rmap != nullptr;
        gemm_tile_fp8_rows<S, true>(rows32, g ? x : x + row0 * H, (int)H, g ? op.xs : op.xs + row0 * (H / 128),
                                    (const uint8_t*)op.wgu + (long)e * 2 * I * H + (long)n0 * H, n0, (int)I,
                                    op.wgus + (long)e * (2 * I / 128) * (H / 128), (int)H, h + row0 * I + n0, (int)I,
                                    op.hs + row0 * (I / 128) + nb, (int)(I / 128), lds,
                                    g ? op.rmap + row0 : nullptr, op.top_k, op.T, hook);
    } else {
        const int n0 = nb * S::BN;
        gemm_tile_fp8_rows<S, false>(rows32, h + row0 * I, (int)I, op.hs + row0 * (I / 128),
                                     (const uint8_t*)op.wd + (long)e * H * I + (long)n0 * I, n0, 0,
                                     op.wds + (long)e * (H / 128) * (I / 128), (int)I, op.y + row0 * H + n0, (int)H,
                                     nullptr, 0, lds, nullptr, 1, 0, hook);
    }
}

template <class Hook>
__device__ __forceinline__ void run_tile(const OpArg& op, int stage, int row0, int rows32, int nb, int e, char* lds,
                                         Hook hook) {
    if (op.cls == CLS_FP8)
        run_tile_fp8<ShapeF8>(op, stage, row0, rows32, nb, e, lds, hook);
    else if (op.cls == CLS_FP8_S)
        run_tile_fp8<ShapeF8S>(op, stage, row0, rows32, nb, e, lds, hook);
    else if (op.cls == CLS_P_BF16)
        run_tile_cls<ShapeP, true>(op, stage, row0, rows32, nb, e, lds, hook);
    else if (op.cls == CLS_D_BF16_S)
        run_tile_cls<ShapeDS, false>(op, stage, row0, rows32, nb, e, lds, hook);
    else
        run_tile_cls<ShapeD, false>(op, stage, row0, rows32, nb, e, lds, hook);
}

// ----------------------------------------------------------------------------- fused combine
// Combine tile t of an op: tokens [t * kCombTokens, ...), 8 per pass, 32 threads
// per token, each thread H/256 16-byte vectors of the token's row (loads of all
// its vectors for one slot are issued together).  Per token and column the
// arithmetic is moe_combine's: fp32 fmaf over the local slots in ascending
// order, then one rounding to the output type.  Outputs are written with
// device-coherent stores, like the tiles' outputs.
constexpr int kCombVec = 6;

__device__ __forceinline__ void st_dev16(void* p, uint4 v) {
    uint64_t* q = (uint64_t*)p;
    __hip_atomic_store(q, (uint64_t)v.x | ((uint64_t)v.y << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(q + 1, (uint64_t)v.z | ((uint64_t)v.w << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void run_combine(const OpArg& op, int t, char* lds, int32_t* status) {
    const int tid = threadIdx.x;
    const int k = op.ck;
    const int tok0 = t * kCombTokens;
    const int ntok = min(kCombTokens, op.ct - tok0);
    int32_t* srow = (int32_t*)lds;                                     // [kCombTokens][k] rows
    float* sw = (float*)(lds + kCombTokens * 32 * sizeof(int32_t));     // [kCombTokens][k] weights
    for (int i = tid; i < ntok * k; i += 256) {
        int r = op.a2r[(size_t)tok0 * k + i];
        if (r >= op.capacity) {
            set_status(status, MOE_ERR_INTERNAL);
            r = -1;
        }
        srow[i] = r;
        sw[i] = op.tw[(size_t)tok0 * k + i];
    }
    __syncthreads();
    const int vecs = op.H >> 3, nv = op.H >> 8, sub = tid & 31;
    const uint4* yp = (const uint4*)op.y;
    for (int p = 0; p < ntok; p += 8) {
        const int tt = p + (tid >> 5);
        if (tt >= ntok) continue;
        for (int u0 = 0; u0 < nv; u0 += kCombVec) {
            float acc[kCombVec][8];
#pragma unroll
            for (int u = 0; u < kCombVec; ++u)
#pragma unroll
                for (int i = 0; i < 8; ++i) acc[u][i] = 0.f;
            for (int j = 0; j < k; ++j) {
                const int r = srow[tt * k + j];
                if (r < 0) continue;
                const float wj = sw[tt * k + j];
                uint4 q[kCombVec];
#pragma unroll
                for (int u = 0; u < kCombVec; ++u)
                    if (u0 + u < nv) q[u] = yp[(size_t)r * vecs + (u0 + u) * 32 + sub];
#pragma unroll
                for (int u = 0; u < kCombVec; ++u) {
                    if (u0 + u >= nv) continue;
                    const uint32_t w4[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        acc[u][2 * i] = fmaf(wj, bf_bits2f(w4[i] & 0xFFFFu), acc[u][2 * i]);
                        acc[u][2 * i + 1] = fmaf(wj, bf_bits2f(w4[i] >> 16), acc[u][2 * i + 1]);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kCombVec; ++u) {
                if (u0 + u >= nv) continue;
                const size_t v = (size_t)(tok0 + tt) * vecs + (u0 + u) * 32 + sub;
                if (op.y_f32) {
                    float* out = (float*)op.yc + v * 8;
                    st_dev16(out, make_uint4(__float_as_uint(acc[u][0]), __float_as_uint(acc[u][1]),
                                             __float_as_uint(acc[u][2]), __float_as_uint(acc[u][3])));
                    st_dev16(out + 4, make_uint4(__float_as_uint(acc[u][4]), __float_as_uint(acc[u][5]),
                                                 __float_as_uint(acc[u][6]), __float_as_uint(acc[u][7])));
                } else {
                    uint4 o;
                    o.x = f2bf_bits(acc[u][0]) | (f2bf_bits(acc[u][1]) << 16);
                    o.y = f2bf_bits(acc[u][2]) | (f2bf_bits(acc[u][3]) << 16);
                    o.z = f2bf_bits(acc[u][4]) | (f2bf_bits(acc[u][5]) << 16);
                    o.w = f2bf_bits(acc[u][6]) | (f2bf_bits(acc[u][7]) << 16);
                    st_dev16((uint4*)op.yc + v, o);
                }
            }
        }
    }
}

// ----------------------------------------------------------------------------- scheduler
// Per-workgroup LDS copy of each op's own-XCD queue (wave 0 only), taken at the
// workgroup's first claim from that queue -- after the claim atomic returned, so
// causally after the op became ACTIVE: the range [lo, lo + cnt) of row tiles and,
// when cnt <= kTabCache, their table entries.  Later claims cost one atomic and
// an LDS read.  lo = -1: not taken yet.
struct TabCache {
    uint64_t ent[MOE_MAX_OPS][kTabCache];
    uint32_t grp[MOE_MAX_OPS][kTabCache];
    int32_t lo[MOE_MAX_OPS];
    int32_t cnt[MOE_MAX_OPS];
};

// Command block written by wave 0 and read by the whole workgroup.
struct Cmd {
    int32_t kind, op, stage, e, row0, rows32, nb, mtile, mblk, rows, t;
    int32_t pre_next;          // op whose next tile wave 0 claims ahead during this tile, or -1
    int32_t q_seen, phases, how;   // the decision's inputs and path (recorded in the trace)
    unsigned long long t_boundary, t_polled, t_claim, t_start, c_start;
};
enum : int32_t { HOW_PREFERRED = 0, HOW_OTHER = 1, HOW_AHEAD = 2, HOW_COMBINE = 3 };

// Lane 0: an op's last tile has committed.  Its outputs were stored
// device-coherent before each tile's commit, and the in-kernel readers of
// DONE (the exit test, a dependent op's start) read no data of the op, so
// DONE itself is a plain store.  With a done word, the acquire takes in every
// other workgroup's writes of this op before the word's system-scope release
// publishes them.
__device__ __forceinline__ void finish_op(const KArgs& a, int o, int total) {
    Hdr* hdr = hdr_of(a.ws);
    OpDyn* d = dyn_of(a.ws) + o;
    uint32_t* dw = a.op[o].done_word;
    if (dw) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const unsigned long long t = wall_ticks();
    __hip_atomic_store(&d->t_done, t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&d->state, (int32_t)ST_DONE, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (dw) st_release_system(dw, 1u);
    if (a.stats) {
        moe_op_stats s;
        s.t_ready = ld_relaxed_agent(&d->t_ready);
        s.t_first = ld_relaxed_agent(&d->t_first);
        s.t_done = t;
        s.t_seen = ld_relaxed_agent(&d->t_seen);
        s.x_moe = ld_relaxed_agent(&d->x_moe);
        s.n_tiles = total;
        s.quota = ld_relaxed_agent(&d->quota);
        s.reserved = 0;
        a.stats[o] = s;
    }
    add_relaxed_agent(&hdr->ops_done, 1);
}

// The words a workgroup reads at a tile boundary to pick its next action
// (wave 0, one op per lane; lane 0 also the header words).  A workgroup
// coming out of a tile issues them right after its K loop, so that their
// round trip overlaps the epilogue; they are then older than the boundary by
// the epilogue's duration.  The raw values are kept (lanes past n_ops read op
// 0) and masked only at the boundary: any arithmetic on them where they are
// issued would make the wave wait for their round trip there.
struct Polls {
    int state, own_claim, own_size, left, phase, stop, q;
    uint32_t abort_v;
};

__device__ __forceinline__ Polls issue_polls(const KArgs& a) {
    const int lane = threadIdx.x;
    const int o_l = lane < a.n_ops ? lane : 0;
    const OpDyn* dyn = dyn_of(a.ws);
    const XQueue* own = xq_of(a.ws, o_l, xcc_id());
    const Hdr* hdr = hdr_of(a.ws);
    Polls p;
    p.state = ld_relaxed_agent(&dyn[o_l].state);
    p.own_claim = ld_relaxed_agent(&own->claim);
    p.own_size = ld_relaxed_agent(&own->size);
    p.left = ld_relaxed_agent(&dyn[o_l].left);
    p.phase = static_of(a.ws)[o_l].phase;
    p.stop = ld_relaxed_agent(&hdr->stop);
    p.q = ld_relaxed_agent(&hdr->quota);
    p.abort_v = a.abort_word ? __hip_atomic_load(a.abort_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) : 0u;
    return p;
}

// At the boundary: lanes past n_ops hold no op.
__device__ __forceinline__ Polls mask_polls(const KArgs& a, Polls p) {
    if ((int)threadIdx.x >= a.n_ops) {
        p.state = ST_DONE;
        p.own_claim = p.own_size = 0;
        p.left = INT32_MIN;
    }
    return p;
}

// Wave 0: the own queue's range and its first kTabCache table and group
// entries (the copies written at instantiation), loaded with one round trip;
// issue() only starts the loads, so a claim issued after them shares their
// round trip, and commit() puts them into the workgroup's LDS cache.
struct TabFill {
    uint64_t ent;
    uint32_t grp;
    int m_lo, n_mt;
    bool on;
};
__device__ __forceinline__ TabFill tab_fill_issue(const KArgs& a, int o, int myx, const TabCache* tab) {
    TabFill f = {};
    f.on = tab->lo[o] < 0;                                     // not cached yet (uniform)
    if (f.on) {
        const OpArg& op = a.op[o];
        const XQueue* qs = xq_of(a.ws, o, myx);
        const int lane = threadIdx.x;
        const char* qt = arr_of(a.ws) + op.qtab_off;
        f.m_lo = ld_relaxed_agent(&qs->m_lo);
        f.n_mt = ld_relaxed_agent(&qs->n_mt);
        f.ent = ld_relaxed_agent((const uint64_t*)qt + myx * kTabCache + lane);
        f.grp = ld_relaxed_agent((const uint32_t*)(qt + kXcds * kTabCache * 8) + myx * kTabCache + lane);
    }
    return f;
}
__device__ __forceinline__ void tab_fill_commit(TabCache* tab, int o, const TabFill& f) {
    if (!f.on) return;
    const int lane = threadIdx.x;
    if (f.n_mt <= kTabCache && lane < f.n_mt) {
        tab->ent[o][lane] = f.ent;
        tab->grp[o][lane] = f.grp;
    }
    if (lane == 0) { tab->lo[o] = f.m_lo; tab->cnt[o] = f.n_mt; }
}

// Wave 0: turn claim t of op o's queue on XCD src into the command block
// (table lookup, validation of the descriptor, GEMM-1 dependency of a GEMM-2
// tile).  The own queue's range and entries are cached in LDS at the first
// claim from it.  Returns, to lane 0, whether the claimed tile was not the own
// queue's last (a next claim from it may succeed).
__device__ __forceinline__ bool take_tile(const KArgs& a, int o, int src, int t, int myx, TabCache* tab, Cmd* cmd,
                  unsigned long long t_boundary, unsigned long long now) {
    const int lane = threadIdx.x;
    Hdr* hdr = hdr_of(a.ws);
    OpDyn* dyn = dyn_of(a.ws);
    bool more = false;
    const OpArg& op = a.op[o];
    const uint64_t* table = (const uint64_t*)(arr_of(a.ws) + op.table_off);
    const uint32_t* grp = (const uint32_t*)(arr_of(a.ws) + op.grp_off);
    int m_lo, n_mt;
    if (src == myx) {
        tab_fill_commit(tab, o, tab_fill_issue(a, o, myx, tab));   // first claim from this op's own queue
        m_lo = tab->lo[o];
        n_mt = tab->cnt[o];
    } else {
        const XQueue* qs = xq_of(a.ws, o, src);
        m_lo = ld_relaxed_agent(&qs->m_lo);
        n_mt = ld_relaxed_agent(&qs->n_mt);
    }
    if (lane == 0) {
        int stage, u, nn, p, mtile, nb;
        sched::queue_pos(t, n_mt, m_lo, op.n1, op.n2, stage, u, nn, p);
        const int lo = tab->lo[o];
        const int cnt = tab->cnt[o];
        const int cg = sched::cache_slot(p, lo, cnt);          // entries of the own queue's row tiles
        const uint32_t g = cg >= 0 ? tab->grp[o][cg] : (p >= 0 && p < op.max_mtiles ? ld_relaxed_agent(grp + p) : 0u);
        sched::group_tile(g, u, nn, m_lo, n_mt, p, mtile, nb);
        const int ce = sched::cache_slot(mtile, lo, cnt);
        const uint64_t ent = ce >= 0 ? tab->ent[o][ce]
                             : (mtile >= 0 && mtile < op.max_mtiles ? ld_relaxed_agent(table + mtile) : 0ull);
        int e, mblk, rows, row0;
        sched::unpack_entry(ent, e, mblk, rows, row0);
        cmd->kind = CMD_TILE; cmd->op = o; cmd->stage = stage;
        cmd->e = e; cmd->mblk = mblk;
        cmd->row0 = row0; cmd->rows = rows; cmd->rows32 = (rows + 31) & ~31;
        // The tile descriptor must address memory inside the op's buffers;
        // if a scheduler invariant broke, stop instead of running the tile.
        if (mtile < 0 || mtile >= op.max_mtiles || e >= op.E || rows < 1 || rows > op.mt || row0 < 0 ||
            (long)row0 + ((rows + 31) & ~31) > (long)op.capacity || nb < 0 || nb >= (stage == 1 ? op.n1 : op.n2)) {
            set_status(a.status, MOE_ERR_INTERNAL);
            st_release_agent(&hdr->stop, 1);
            cmd->kind = CMD_EXIT;
        }
        cmd->nb = nb; cmd->mtile = mtile; cmd->t = t;
        cmd->t_boundary = t_boundary;
        cmd->t_polled = now;
        cmd->t_claim = wall_ticks();
        if (t == 0) {
            unsigned long long zero = 0;
            __hip_atomic_compare_exchange_strong(&dyn[o].t_first, &zero, cmd->t_claim, __ATOMIC_RELAXED,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (stage == 2 && cmd->kind == CMD_TILE) {            // GEMM-1 of this row tile must be committed
            const int32_t* g1 = (const int32_t*)(arr_of(a.ws) + op.g1_off) + mtile;
            int64_t spins = 0;
            while (ld_relaxed_agent(g1) < op.n1) {
                if (++spins > a.spin_limit || ld_relaxed_agent(&hdr->stop)) {
                    set_status(a.status, MOE_ERR_TIMEOUT);
                    st_release_agent(&hdr->stop, 1);
                    cmd->kind = CMD_EXIT;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        cmd->t_start = wall_ticks();
        cmd->c_start = __builtin_amdgcn_s_memtime();
        more = src == myx && t + 1 < n_mt * (op.n1 + op.n2);
    }
    return more;
}

// Wave 0: combine tile t of op o (stage 3) into the command block.
__device__ void take_combine(int o, int t, Cmd* cmd, unsigned long long t_boundary, unsigned long long now) {
    if (threadIdx.x == 0) {
        cmd->kind = CMD_TILE; cmd->op = o; cmd->stage = 3; cmd->t = t;
        cmd->e = -1; cmd->mblk = t; cmd->row0 = 0; cmd->rows = 0; cmd->rows32 = 0; cmd->nb = 0; cmd->mtile = -1;   // trace: mblk = tile
        cmd->pre_next = -1;
        cmd->t_boundary = t_boundary;
        cmd->t_polled = now;
        cmd->t_claim = wall_ticks();
        cmd->t_start = cmd->t_claim;
        cmd->c_start = __builtin_amdgcn_s_memtime();
    }
}

// Whether a workgroup may claim its next tile of an op of this phase ahead,
// during the current tile: only in its preferred phase (decode below q', or
// any workgroup when the launch holds no prefill op), and for prefill only if
// it can never be asked to prefer decode (index >= every possible q'), so a
// claim made ahead never delays a decode tile or holds one beyond the quota.
__device__ __forceinline__ bool pre_allowed(const KArgs& a, int wg, int q, int phase) {
    return phase == MOE_DECODE ? (wg < q || a.pre_dec_all) : wg >= a.pre_wg;
}
__device__ __forceinline__ int phase_of(const KArgs& a, int o) { return a.op[o].phase; }

// Wave 0 at a tile boundary: commit the previous tile (if any), decide with
// the polled words (pre, issued after the previous tile's K loop, when
// have_pre; else read now), claim, and only then wait for the commit's
// completion count, so the commit and the claim share one round trip.
template <bool COMB>
__device__ __forceinline__ void boundary(const KArgs& a, uint64_t t0, int wg, Cmd* cmd, bool have_prev, int64_t& idle,
                         TabCache* tab, bool have_pre, Polls pre, int pre_t, const int32_t* n3s, int& n_traced) {
    const int lane = threadIdx.x;
    Hdr* hdr = hdr_of(a.ws);
    OpDyn* dyn = dyn_of(a.ws);
    const OpStatic* sta = static_of(a.ws);
    // The command block still describes the tile just run (it is rewritten
    // only below), so the previous tile is read from LDS rather than kept in
    // registers across the tile.
    Cmd prev;
    if (have_prev) prev = *cmd;
    if (lane == 0) cmd->pre_next = -1;
    const unsigned long long t_boundary = wall_ticks();
    const Polls pl = mask_polls(a, have_pre ? pre : issue_polls(a));

    // 1. commit: count the tile (its device-coherent stores have completed).
    //    Both counters are bumped with atomics whose result is not used, so the
    //    boundary never waits for their round trip; whether the op is complete
    //    is read from the polled counts (step 2b), by whichever workgroup
    //    first sees them full.
    unsigned long long t_end = 0, c_end = 0;
    if (have_prev && lane == 0) {
        t_end = wall_ticks();
        c_end = __builtin_amdgcn_s_memtime();
        if (prev.stage == 1) {
            int32_t* g1 = (int32_t*)(arr_of(a.ws) + a.op[prev.op].g1_off);
            __hip_atomic_fetch_add(g1 + prev.mtile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __hip_atomic_fetch_add(&dyn[prev.op].left, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // 3. trace the previous tile, into this workgroup's own block of records
    //    (no shared counter, so tracing adds no round trip to a boundary)
    auto finish_prev = [&]() {
        if (have_prev && lane == 0) {
            if (a.trace) {
                const int64_t idx = (int64_t)wg * a.trace_per_wg + n_traced;
                if (n_traced < a.trace_per_wg) {
                    ++n_traced;
                    moe_trace_rec r;
                    r.op = (int16_t)prev.op; r.stage = (int16_t)prev.stage; r.wg = (int16_t)wg;
                    r.xcc = (int16_t)xcc_id(); r.expert = prev.e; r.mblk = prev.mblk; r.nblk = (int16_t)prev.nb;
                    r.rows = (int16_t)prev.rows; r.quota_seen = (int16_t)prev.q_seen;
                    r.phases_seen = (uint8_t)prev.phases; r.how = (uint8_t)prev.how;
                    r.t_boundary = prev.t_boundary; r.t_polled = prev.t_polled;
                    r.t_claim = prev.t_claim; r.t_start = prev.t_start; r.t_end = t_end;
                    r.c_start = prev.c_start; r.c_end = c_end;
                    a.trace[idx] = r;
                }
            }
        }
    };

    // 2. stop conditions (polled)
    int state = pl.state;
    const int own_claim = pl.own_claim, own_size = pl.own_size;
    const int o_l = lane < a.n_ops ? lane : 0;
    const int phase = pl.phase;
    const int myx = xcc_id();
    int stop = 0;
    if (lane == 0) {
        stop = pl.stop;
        if (!stop && pl.abort_v != 0u) {
            set_status(a.status, MOE_ERR_ABORTED);
            st_release_agent(&hdr->stop, 1);
            stop = 1;
        }
        if (!stop && idle > a.spin_limit) {                    // nothing claimable for too long
            set_status(a.status, MOE_ERR_TIMEOUT);
            st_release_agent(&hdr->stop, 1);
            stop = 1;
        }
    }
    if (__shfl(stop, 0, 64)) {
        finish_prev();
        if (lane == 0) cmd->kind = CMD_EXIT;
        return;
    }
    int q = __shfl(pl.q, 0, 64);
    // 2b. an op whose every tile had committed when polled is finished by the
    //     workgroup that wins its ACTIVE -> FINISHING transition (left only
    //     grows and is 0 only once the last tile committed, so a stale poll can
    //     only delay this, never fire it early)
    //     With a fused combine, the op's GEMM tiles are all committed when left
    //     reaches -n3: then it turns COMBINING, and its combine tiles can be
    //     claimed (every y_perm row they read was stored before its commit).
    const int n3_l = COMB && lane < a.n_ops ? n3s[lane] : 0;
    //     The polls were issued before this workgroup's commit: if they show
    //     its op one tile short, that tile is this workgroup's own and the
    //     commit just issued completes the op (no further poll needed).
    const bool own_last = have_prev && prev.stage != 3 && lane == prev.op && pl.left == -1;
    const uint64_t fmask = __ballot((pl.left == 0 || own_last) &&
                                    ((state == ST_ACTIVE && n3_l == 0) || (COMB && state == ST_COMBINING)));
    const uint64_t cmask = COMB ? __ballot(state == ST_ACTIVE && n3_l > 0 && pl.left == -n3_l) : 0ull;
    if (fmask | cmask) {
        int won = 0;
        if ((fmask >> lane) & 1) won = atomicCAS(&dyn[lane].state, state, ST_FINISHING) == state;
        if (COMB && ((cmask >> lane) & 1)) atomicCAS(&dyn[lane].state, ST_ACTIVE, ST_COMBINING);
        uint64_t wmask = __ballot(won);
        while (wmask) {                                              // wave-uniform loop
            const int o = __ffsll((long long)wmask) - 1;
            wmask &= wmask - 1;
            if (lane == 0) finish_op(a, o, ld_relaxed_agent(&dyn[o].total));
        }
        if ((fmask >> lane) & 1) state = ST_DONE;                   // finished here or by its winner
        if (COMB && ((cmask >> lane) & 1)) state = ST_COMBINING;    // turned here or by another workgroup
    }
    if (__ballot(state != ST_DONE) == 0) {
        // every op was DONE when polled (or was finished just above)
        finish_prev();
        if (lane == 0) cmd->kind = CMD_EXIT;
        return;
    }
    const uint64_t now = wall_ticks();
    // phases with claimable work in the polls this decision uses (recorded in the trace)
    bool active = state == ST_ACTIVE || (COMB && state == ST_COMBINING);
    uint64_t dmask = __ballot(active && phase == MOE_DECODE);
    uint64_t pmask = __ballot(active && phase == MOE_PREFILL);
    int phases_seen = (dmask ? 1 : 0) | (pmask ? 2 : 0);

    // 3b. a claim made ahead during the previous tile (the hook claimed in this
    //     XCD's queue of op prev.pre_next): take it if it landed inside the queue
    const int pre_op_u = have_prev ? prev.pre_next : -1;
    if (pre_op_u >= 0) {
        const int pt = __shfl(pre_t, 0, 64);
        if (pt < __shfl(own_size, pre_op_u, 64)) {
            finish_prev();
            const bool more = take_tile(a, pre_op_u, myx, pt, myx, tab, cmd, t_boundary, now);
            if (lane == 0) {
                cmd->pre_next = more && pre_allowed(a, wg, q, phase_of(a, pre_op_u)) ? pre_op_u : -1;
                cmd->q_seen = q; cmd->phases = phases_seen; cmd->how = HOW_AHEAD;
            }
            idle = 0;
            return;
        }
    }

    // 4. ready signals of waiting operation templates -> instantiate one of them.
    //    A decode template is instantiated only by a workgroup below the
    //    smallest q' the launch can produce, which therefore prefers decode and
    //    takes the op's first tile at its very next boundary: a decode op waits
    //    for one tile boundary of those workgroups plus its instantiation.
    //    A template built ahead (4b) needs no instantiation: the same
    //    workgroups activate it and claim its first tile in the same boundary.
    //    The release condition is also read by a workgroup that may build a
    //    template ahead (4b), so that one already released is left to the
    //    workgroups that instantiate it at once.
    bool ready = false;
    const bool built = is_built(state);
    const bool may_inst = phase == MOE_PREFILL || a.inst_wg == 0 || wg < a.inst_wg;
    const bool may_build = wg >= a.pre_wg && state == ST_WAIT && sta[o_l].rel_word == nullptr;
    if ((state == ST_WAIT || built) && (may_inst || may_build)) {
        ready = true;
        const uint32_t* rw = sta[o_l].rel_word;
        if (rw) ready = __hip_atomic_load(rw, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0u;
        if (ready && sta[o_l].rel_after >= 0) ready = now >= t0 + (uint64_t)sta[o_l].rel_after;
        const int dep = sta[o_l].dep;
        if (ready && dep >= 0) {
            ready = ld_relaxed_agent(&dyn[dep].state) == ST_DONE &&
                    now >= ld_relaxed_agent(&dyn[dep].t_done) + (uint64_t)sta[o_l].gap;
        }
    }
    const bool released = ready;                          // (read where may_inst or may_build)
    ready = ready && may_inst;
    // 4a. activation of a built template: one transition of its state word.
    //     Its queue words and table entries reached the coherence point before
    //     the word turned BUILT, so every claim that follows the transition
    //     finds them.  An op with no row tiles finishes here (or turns
    //     COMBINING: its combine tiles write zeros).
    const uint64_t amask = __ballot(ready && built);
    if (amask) {
        const int o = __ffsll((long long)amask) - 1;
        int to = 0;
        if (lane == o) {
            const bool empty = (state >> 4) & 1;
            const int next = !empty ? ST_ACTIVE : (n3_l > 0 ? ST_COMBINING : ST_FINISHING);
            if (atomicCAS(&dyn[o].state, state, next) == state) {
                to = next;
                __hip_atomic_store(&dyn[o].t_seen, (unsigned long long)now, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&dyn[o].t_ready, (unsigned long long)now, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (empty) {
                    __hip_atomic_store(&dyn[o].t_first, (unsigned long long)now, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (next == ST_FINISHING) finish_op(a, o, 0);
                } else if (phase == MOE_DECODE) {
                    __hip_atomic_store(&hdr->quota, state >> 5, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        }
        to = __shfl(to, o, 64);
        const int qd = __shfl(state >> 5, o, 64);
        if (to != 0) {
            if (lane == o) state = to == ST_FINISHING ? ST_DONE : to;
            if (to == ST_ACTIVE && phase_of(a, o) == MOE_DECODE) q = qd;
            active = state == ST_ACTIVE || (COMB && state == ST_COMBINING);
            dmask = __ballot(active && phase == MOE_DECODE);
            pmask = __ballot(active && phase == MOE_PREFILL);
            phases_seen = (dmask ? 1 : 0) | (pmask ? 2 : 0);
            idle = 0;
        }
    }
    const uint64_t rmask = __ballot(ready && !built);
    if (rmask) {
        const int o = __ffsll((long long)rmask) - 1;
        int won = 0;
        if (lane == o) {
            won = atomicCAS(&dyn[o].state, ST_WAIT, ST_INIT) == ST_WAIT;
            if (won) __hip_atomic_store(&dyn[o].t_seen, (unsigned long long)now, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (__ballot(won)) {
            finish_prev();
            if (lane == 0) { cmd->kind = CMD_INST; cmd->op = o; cmd->stage = 1; }
            idle = 0;
            return;
        }
    }
    // 4b. build ahead: a template whose inputs were in place at the launch (no
    //     release word) is built before its ready signal, by a workgroup that
    //     never prefers decode, and waits BUILT.
    if (wg >= a.pre_wg) {
        const uint64_t bmask = __ballot(may_build && !released);
        if (bmask) {
            const int o = __ffsll((long long)bmask) - 1;
            int won = 0;
            if (lane == o) won = atomicCAS(&dyn[o].state, ST_WAIT, ST_INIT) == ST_WAIT;
            if (__ballot(won)) {
                finish_prev();
                if (lane == 0) { cmd->kind = CMD_INST; cmd->op = o; cmd->stage = 0; }
                idle = 0;
                return;
            }
        }
    }

    // 5. claim: decode first on workgroups below q', prefill first elsewhere;
    //    within a phase: the own XCD's queue first, then steal from the others
    const uint64_t combining = COMB ? __ballot(state == ST_COMBINING) : 0ull;
    const uint64_t own_avail = __ballot(active && own_claim < own_size);
    const bool prefer_decode = a.split ? wg < a.pre_wg : wg < q;
    const uint64_t order[2] = {prefer_decode ? dmask : pmask, prefer_decode ? pmask : dmask};
    for (int p = 0; p < (a.split ? 1 : 2); ++p) {                   // a static partition never borrows
        uint64_t m = order[p];
        while (m) {                                                  // wave-uniform loop
            const int o = __ffsll((long long)m) - 1;
            m &= m - 1;
            int src = -1, t = 0;
            if (COMB && ((combining >> o) & 1)) {                   // one shared queue of combine tiles
                if (lane == 0) t = atomicAdd(&dyn[o].cclaim, 1);
                t = __shfl(t, 0, 64);
                if (t >= n3s[o]) continue;
                finish_prev();
                take_combine(o, t, cmd, t_boundary, now);
                if (lane == 0) { cmd->q_seen = q; cmd->phases = phases_seen; cmd->how = HOW_COMBINE; }
                idle = 0;
                return;
            }
            if ((own_avail >> o) & 1) {                             // own queue
                const TabFill f = tab_fill_issue(a, o, myx, tab);   // shares the claim's round trip
                if (lane == 0) t = atomicAdd(&xq_of(a.ws, o, myx)->claim, 1);
                t = __shfl(t, 0, 64);
                tab_fill_commit(tab, o, f);
                if (t < __shfl(own_size, o, 64)) src = myx;
            }
            // steal: the queue with most tiles left; a lost race tries again,
            // so the op is left only once every one of its queues is empty.
            // A failed claim means that queue's counter passed its size for
            // good, so there are at most kXcds failures: the loop ends.
            while (src < 0) {
                const XQueue* qx = xq_of(a.ws, o, lane & (kXcds - 1));
                int left = 0;
                if (lane < kXcds) left = ld_relaxed_agent(&qx->size) - ld_relaxed_agent(&qx->claim);
                int best = left, who = lane;
#pragma unroll
                for (int off = 4; off >= 1; off >>= 1) {             // max over lanes 0..7
                    const int ob = __shfl_xor(best, off, 64), ow = __shfl_xor(who, off, 64);
                    if (ob > best || (ob == best && ow < who)) { best = ob; who = ow; }
                }
                best = __shfl(best, 0, 64);
                who = __shfl(who, 0, 64);
                if (best <= 0) break;
                if (lane == 0) t = atomicAdd(&xq_of(a.ws, o, who)->claim, 1);
                t = __shfl(t, 0, 64);
                int sz = 0;
                if (lane == 0) sz = ld_relaxed_agent(&xq_of(a.ws, o, who)->size);
                if (t < __shfl(sz, 0, 64)) src = who;
            }
            if (src < 0) continue;
            finish_prev();
            const bool more = take_tile(a, o, src, t, myx, tab, cmd, t_boundary, now);
            if (lane == 0) {
                cmd->pre_next = more && pre_allowed(a, wg, q, phase_of(a, o)) ? o : -1;
                cmd->q_seen = q; cmd->phases = phases_seen; cmd->how = p == 0 ? HOW_PREFERRED : HOW_OTHER;
            }
            idle = 0;
            return;
        }
    }
    finish_prev();
    // Nothing claimable, every op activated and every queue of every active
    // op found empty above: no tile can become claimable here any more (no
    // template waits for its release, no combine tiles will follow), so the
    // workgroup leaves now rather than polling until the last op is finished
    // by the workgroups still running its tiles.
    // The polls predate this boundary's commit, so that commit may have been
    // the last of its op: once it has completed, an op whose count reads full
    // is finished here (unless another workgroup wins it), since no
    // workgroup may be left to see it full later.
    if (!COMB && !a.split && __ballot(state == ST_WAIT || state == ST_INIT || is_built(state)) == 0) {
        wait_own_stores();
        int won = 0;
        if (lane < a.n_ops && state == ST_ACTIVE && ld_relaxed_agent(&dyn[lane].left) == 0)
            won = atomicCAS(&dyn[lane].state, ST_ACTIVE, ST_FINISHING) == ST_ACTIVE;
        uint64_t wmask = __ballot(won);
        while (wmask) {                                              // wave-uniform loop
            const int o = __ffsll((long long)wmask) - 1;
            wmask &= wmask - 1;
            if (lane == 0) finish_op(a, o, ld_relaxed_agent(&dyn[o].total));
        }
        if (lane == 0) cmd->kind = CMD_EXIT;
        return;
    }
    if (lane == 0) cmd->kind = CMD_IDLE;
    ++idle;
}

// Whole workgroup, first half of building an op's row tiles: its counts and
// offsets into LDS and scan[e] = the first row tile of expert e (Eq. (3) row
// tiles per expert); *s_total = x_moe, *s_bad = 1 if the offsets or counts do
// not fit the op's buffers.  Ends with the workgroup synchronised.
__device__ void scan_row_tiles(const OpArg& op, int32_t* scan, int32_t* s_cnt, int32_t* s_off, int32_t* s_total,
                               int32_t* s_bad) {
    // one round trip for the op's inputs: counts and offsets together, into LDS
    for (int e = threadIdx.x; e < op.E; e += 256) {
        const int c = op.counts[e], off = op.offsets[e];
        s_cnt[e] = c;
        s_off[e] = off;
        scan[e] = sched::row_tiles(c, op.mt);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
        // exclusive scan of the row-tile counts by wave 0: each lane sums a run
        // of up to 16 experts, the run totals are scanned across the wave
        const int lane = threadIdx.x, per = (op.E + 63) / 64, e0 = lane * per;
        const int e1 = e0 + per < op.E ? e0 + per : op.E;
        int sum = 0;
        for (int e = e0; e < e1; ++e) sum += scan[e];
        int incl = sum;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int v = __shfl_up(incl, d, 64);
            if (lane >= d) incl += v;
        }
        int run = incl - sum;
        for (int e = e0; e < e1; ++e) { const int v = scan[e]; scan[e] = run; run += v; }
        if (lane == 63) *s_total = incl;
        if (lane == 0) *s_bad = 0;
    }
    __syncthreads();
    // every expert's segment must fit the op's buffers and tables
    for (int e = threadIdx.x; e < op.E; e += 256) {
        const int c = s_cnt[e], nt = sched::row_tiles(c, op.mt), off = s_off[e];
        const int nb32 = (c + kSegAlign - 1) / kSegAlign;        // 32-row blocks of the segment
        if (scan[e] + nt > op.max_mtiles || off < 0 || (long)off + (long)nb32 * kSegAlign > op.capacity) *s_bad = 1;
    }
    __syncthreads();
}

// Whole workgroup, second half: one thread per row tile stores its table
// entry (expert, row blocks of near-equal height, first row) and its
// weight-sharing group entry.  With queue cuts (cut[x] = first row tile of
// queue x, cut[kXcds] = x_moe), a row tile among the first kTabCache of its
// queue is also stored in that queue's block of copies, which a workgroup
// loads together with its first claim from the queue.
__device__ void store_row_tiles(const OpArg& op, uint64_t* table, uint32_t* grp, int gmax, const int32_t* scan,
                                const int32_t* s_cnt, const int32_t* s_off, int total, const int32_t* cut,
                                uint64_t* qent, uint32_t* qgrp) {
    total = total < op.max_mtiles ? total : op.max_mtiles;
    for (int p = threadIdx.x; p < total; p += 256) {
        uint64_t ent;
        uint32_t g;
        if (!sched::row_tile_entry(scan, s_cnt, s_off, op.E, total, op.mt, gmax, p, ent, g)) continue;
        // device-coherent stores: a reader on any XCD that has seen the op
        // ACTIVE reads them from the coherence point
        __hip_atomic_store(table + p, ent, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(grp + p, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (cut) {
            int x = 0;
            for (int y = 1; y < kXcds; ++y)
                if (cut[y] <= p) x = y;                         // the last queue starting at or before p
            const int slot = p - cut[x];
            if (slot < kTabCache) {
                __hip_atomic_store(qent + x * kTabCache + slot, ent, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(qgrp + x * kTabCache + slot, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
}

// Whole workgroup: the row-tile table and group entries of an op (the plain
// grids' planning step).
__device__ void build_row_tiles(const OpArg& op, uint64_t* table, uint32_t* grp, int gmax, int32_t* scan,
                                int32_t* s_cnt, int32_t* s_off, int32_t* s_total, int32_t* s_bad) {
    scan_row_tiles(op, scan, s_cnt, s_off, s_total, s_bad);
    store_row_tiles(op, table, grp, gmax, scan, s_cnt, s_off, *s_total, nullptr, nullptr, nullptr);
}

// Whole workgroup: builds op o's row tiles, queues and counters; with act,
// the op then turns ACTIVE (its ready signal was seen), else it waits BUILT
// for its activation (4a in boundary), which sets the decode quota.
__device__ __forceinline__ void instantiate(const KArgs& a, int o, bool act, int32_t* scan, int32_t* s_cnt,
                                            int32_t* s_off) {
    const OpArg& op = a.op[o];
    OpDyn* d = dyn_of(a.ws) + o;
    if (op.rel) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");  // system scope: peer-written inputs
    const int gmax = a.gmax;
    __shared__ int32_t s_total, s_bad, s_cut[kXcds + 1];
    scan_row_tiles(op, scan, s_cnt, s_off, &s_total, &s_bad);
    // Queue cuts: cut x (1..kXcds-1) is the group boundary nearest to x/kXcds
    // of the row tiles (ties: the lower one), so no group spans two queues;
    // cuts are non-decreasing in x.
    const int xm = s_total < op.max_mtiles ? s_total : op.max_mtiles;
    if (threadIdx.x < kXcds + 1)
        s_cut[threadIdx.x] = threadIdx.x == 0 ? 0 : threadIdx.x == kXcds ? xm : sched::queue_cut(threadIdx.x, scan, op.E, xm, gmax);
    __syncthreads();
    const bool bad = s_bad != 0;
    if (!bad) {
        char* arr = arr_of(a.ws);
        store_row_tiles(op, (uint64_t*)(arr + op.table_off), (uint32_t*)(arr + op.grp_off), gmax, scan, s_cnt, s_off,
                        xm, s_cut, (uint64_t*)(arr + op.qtab_off), (uint32_t*)(arr + op.qtab_off + kXcds * kTabCache * 8));
    }
    int qd = 0;
    if (threadIdx.x == 0 && !bad) {
        Hdr* hdr = hdr_of(a.ws);
        if (op.phase == MOE_DECODE) {
            qd = decode_quota(a.q, xm, a.x_star, a.q_max, a.c);
            if (act) __hip_atomic_store(&hdr->quota, qd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __hip_atomic_store(&d->x_moe, xm, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // the commit counter is set before any queue can hand out a tile
        __hip_atomic_store(&d->total, xm * (op.n1 + op.n2) + op.n3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&d->left, -(xm * (op.n1 + op.n2) + op.n3), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (int x = 0; x < kXcds; ++x) {                      // contiguous row-tile ranges, cut between groups
            XQueue* qx = xq_of(a.ws, o, x);
            const int lo = s_cut[x], hi = s_cut[x + 1];
            __hip_atomic_store(&qx->m_lo, lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&qx->n_mt, hi - lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&qx->size, (hi - lo) * (op.n1 + op.n2), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __hip_atomic_store(&d->quota, qd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // Every wave's table entries and wave 0's queue words have reached the
    // coherence point before the barrier that precedes ACTIVE; no L2
    // write-back is needed (an agent-scope release would write back the XCD's
    // whole L2, dirtied by the kernels before).
    wait_own_stores();
    __syncthreads();
    if (threadIdx.x == 0) {
        if (bad) {
            set_status(a.status, MOE_ERR_CAPACITY);
            st_release_agent(&hdr_of(a.ws)->stop, 1);
            return;
        }
        if (!act) {
            __hip_atomic_store(&d->state, built_word(xm, qd), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
        const unsigned long long t = wall_ticks();
        __hip_atomic_store(&d->t_ready, t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (xm == 0) {                                   // nothing routed here: done at once
            __hip_atomic_store(&d->t_first, t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (op.n3 > 0) st_release_agent(&d->state, (int32_t)ST_COMBINING);   // its combine writes zeros
            else finish_op(a, o, 0);
        } else {
            __hip_atomic_store(&d->state, (int32_t)ST_ACTIVE, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// COMB: some op of the launch has a fused combine (a separate instance, so the
// plain kernel's register allocation does not carry the combine path).
template <bool COMB>
__global__ __launch_bounds__(256, 1) void apk_kernel(const KArgs a) {
    extern __shared__ __align__(16) char lds[];
    __shared__ Cmd cmd;
    __shared__ int32_t scan[1024];
    __shared__ int32_t s_cnt[1024], s_off[1024];              // instantiation: the op's counts and offsets
    __shared__ unsigned long long s_t0;
    __shared__ TabCache tab;
    __shared__ int32_t s_n3[MOE_MAX_OPS];                     // combine tiles per op
    const int tid = threadIdx.x;
    const int wg = blockIdx.x;
    if (tid < MOE_MAX_OPS) {
        tab.lo[tid] = -1;
        tab.cnt[tid] = 0;
        s_n3[tid] = tid < a.n_ops ? a.op[tid].n3 : 0;
    }
    if (tid == 0) {
        const unsigned long long now = wall_ticks();
        const unsigned long long prev = atomicCAS(&hdr_of(a.ws)->t0, 0ull, now);
        s_t0 = prev ? prev : now;
        if (wg == 0) __hip_atomic_store(&hdr_of(a.ws)->n_wg, (int32_t)gridDim.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    const uint64_t t0 = s_t0;
    int64_t idle = 0;
    int n_traced = 0;                                         // lane 0: records written to this workgroup's block
    bool have_prev = false;
    bool have_pre = false;                                    // polls issued during the last tile (GEMM tiles only)
    Polls polls = {};                                         // wave 0: issued after the last tile's K loop
    int pre_t = 0;                                            // lane 0: a claim issued ahead, during the tile
    for (;;) {
        if (tid < 64) boundary<COMB>(a, t0, wg, &cmd, have_prev, idle, &tab, have_pre, polls, pre_t, s_n3, n_traced);
        __syncthreads();
        const int kind = cmd.kind;
        have_prev = false;
        have_pre = false;                                     // set again only by a GEMM tile's hook
        if (kind == CMD_EXIT) {
            if (tid == 0)
                __hip_atomic_fetch_max(&hdr_of(a.ws)->t_exit, (unsigned long long)wall_ticks(), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            if (tid == 0 && a.trace && n_traced < a.trace_per_wg) {      // end of this workgroup's records
                moe_trace_rec r = {};
                r.op = -1;
                r.wg = (int16_t)wg;
                a.trace[(int64_t)wg * a.trace_per_wg + n_traced] = r;
            }
            break;
        }
        if (kind == CMD_IDLE) {
            __builtin_amdgcn_s_sleep(8);
            __syncthreads();                                  // cmd is rewritten next iteration
            continue;
        }
        if (kind == CMD_INST) {
            const int o = __builtin_amdgcn_readfirstlane(cmd.op);
            const bool act = __builtin_amdgcn_readfirstlane(cmd.stage) != 0;
            __syncthreads();
            instantiate(a, o, act, scan, s_cnt, s_off);
            __syncthreads();
            continue;
        }
        const int o = __builtin_amdgcn_readfirstlane(cmd.op);
        const int stage = __builtin_amdgcn_readfirstlane(cmd.stage);
        const int row0 = __builtin_amdgcn_readfirstlane(cmd.row0);
        const int rows32 = __builtin_amdgcn_readfirstlane(cmd.rows32);
        const int nb = __builtin_amdgcn_readfirstlane(cmd.nb);
        const int e = __builtin_amdgcn_readfirstlane(cmd.e);
        const int ct = __builtin_amdgcn_readfirstlane(cmd.t);
        __syncthreads();                                      // every thread has read cmd
        if (COMB && stage == 3) {
            run_combine(a.op[o], ct, lds, a.status);
        } else {
            have_pre = true;
            run_tile(a.op[o], stage, row0, rows32, nb, e, lds, [&]() {
                // (both results are assigned on every path, so neither stays live across the K loop)
                Polls p = {};
                int t_ahead = 0;
                if (tid < 64) {
                    p = issue_polls(a);
                    // claim the next tile of the same op ahead; its round trip overlaps the epilogue
                    const int pn = cmd.pre_next;                  // written by this wave at the boundary
                    if (tid == 0 && pn >= 0) t_ahead = atomicAdd(&xq_of(a.ws, pn, xcc_id())->claim, 1);
                }
                polls = p;
                pre_t = t_ahead;
            });
        }
        // The commit counts on every wave's stores having reached the L2; the barrier
        // does not wait for global stores, so each wave first waits for its own.
        wait_own_stores();
        __syncthreads();
        have_prev = true;
    }
}

struct ClassInfo {
    int bm, bn, bk;            // tallest row tile (Eq. 3's M_t), output columns, K step
};
ClassInfo class_info(int cls) {
    if (is_fp8_cls(cls)) return ClassInfo{ShapeF8::BM, ShapeF8::BN, ShapeF8::BK};
    return cls == CLS_P_BF16 ? ClassInfo{ShapeP::BM, ShapeP::BN, ShapeP::BK} : ClassInfo{ShapeD::BM, ShapeD::BN, ShapeD::BK};
}
int class_of(int phase, int dtype) {
    if (dtype == MOE_FP8_E4M3) return CLS_FP8;
    return phase == MOE_PREFILL ? CLS_P_BF16 : CLS_D_BF16;
}

// Per op: a row-tile table (8 bytes per row tile), GEMM-1 counters and group
// entries (4 bytes per row tile each), each padded to 256 bytes so no L2 line
// is shared between ops, then per queue the copies of its first kTabCache
// table and group entries.
constexpr size_t kQtabBytes = (size_t)kXcds * kTabCache * (8 + 4);
static_assert(kQtabBytes % 256 == 0, "whole L2 lines");
size_t op_array_bytes(int capacity, int mt, size_t* table_bytes, size_t* group_bytes) {
    const size_t mm = (size_t)((capacity + mt - 1) / mt) + 1;
    const size_t tb = (mm * 8 + 255) & ~(size_t)255;
    const size_t gb = (mm * 4 + 255) & ~(size_t)255;
    if (table_bytes) *table_bytes = tb;
    if (group_bytes) *group_bytes = gb;
    return tb + 2 * gb + kQtabBytes;
}

size_t ws_bytes_for(const moe_op_desc* ops, int n_ops) {
    size_t bytes = kArraysOff;
    for (int o = 0; o < n_ops; ++o) bytes += op_array_bytes(ops[o].capacity, kSegAlign, nullptr, nullptr);
    return (bytes + 255) & ~(size_t)255;
}

}  // namespace

extern "C" int32_t moe_ffn_row_align(moe_phase_t phase, moe_dtype_t dtype) {
    if (phase != MOE_PREFILL && phase != MOE_DECODE) return -1;
    if (dtype != MOE_BF16 && dtype != MOE_FP8_E4M3) return -2;
    (void)class_info(class_of(phase, dtype));
    return kSegAlign;
}

extern "C" moe_status_t moe_ffn_tile_shape(moe_phase_t phase, moe_dtype_t dtype, int32_t* bm, int32_t* bn,
                                           int32_t* bk) {
    if ((phase != MOE_PREFILL && phase != MOE_DECODE) || (dtype != MOE_BF16 && dtype != MOE_FP8_E4M3))
        return moeapk_host::fail(MOE_ERR_UNSUPPORTED, "moe_ffn_tile_shape: phase %d dtype %d", phase, dtype);
    const ClassInfo ci = class_info(class_of(phase, dtype));
    if (bm) *bm = ci.bm;
    if (bn) *bn = ci.bn;
    if (bk) *bk = ci.bk;
    return MOE_OK;
}

extern "C" size_t moe_ffn_workspace_bytes(const moe_op_desc* ops, int32_t n_ops, const moe_sched_config* cfg) {
    (void)cfg;
    if (!ops || n_ops < 1 || n_ops > MOE_MAX_OPS) return 0;
    return ws_bytes_for(ops, n_ops);
}

namespace {

// Checks every op descriptor and fills the kernel's per-op arguments and the
// init kernel's readiness fields; off = the ops' array bytes.  Shared by the
// persistent launch and the plain-grid baseline.
// prefill_rows: 0 or 192 = the tall prefill tiles; 128 = bf16 prefill ops run the 128-row tile class.
moe_status_t fill_ops(const moe_op_desc* ops, int32_t n_ops, int wc_khz, KArgs& a, InitArgs& ia, size_t& off,
                      int prefill_rows = 0) {
    using moeapk_host::fail;
    off = 0;                                          // bytes from the arrays base
    bool with_prefill = false;                        // bf16 decode tiles then stream their weights (ShapeDS)
    for (int o = 0; o < n_ops; ++o) with_prefill |= ops[o].phase == MOE_PREFILL;
    for (int o = 0; o < n_ops; ++o) {
        const moe_op_desc& d = ops[o];
        if (d.phase != MOE_PREFILL && d.phase != MOE_DECODE) return fail(MOE_ERR_INVALID_ARG, "op %d: bad phase %d", o, d.phase);
        if (d.dtype != MOE_BF16 && d.dtype != MOE_FP8_E4M3)
            return fail(MOE_ERR_UNSUPPORTED, "op %d: dtype %d not supported by the FFN kernel", o, d.dtype);
        if (d.weight_layout != MOE_LAYOUT_PACKED)
            return fail(MOE_ERR_UNSUPPORTED, "op %d: weights must be in MOE_LAYOUT_PACKED (moe_pack_weights)", o);
        int cls = class_of(d.phase, d.dtype);
        if (cls == CLS_P_BF16 && prefill_rows == 128) cls = CLS_D_BF16;
        else if (cls == CLS_D_BF16 && with_prefill) cls = CLS_D_BF16_S;
        else if (cls == CLS_FP8 && d.phase == MOE_DECODE && with_prefill) cls = CLS_FP8_S;
        const ClassInfo ci = class_info(cls);
        if (d.E_local < 1 || d.E_local > 1024) return fail(MOE_ERR_UNSUPPORTED, "op %d: E_local=%d outside [1,1024]", o, d.E_local);
        // H and I are the K of a GEMM (whole pairs of K steps) and split into whole output tiles
        if (d.H < ci.bn || d.H % ci.bn != 0 || d.H % (2 * ci.bk) != 0 || d.H % 256 != 0)
            return fail(MOE_ERR_UNSUPPORTED, "op %d: H=%d must be a positive multiple of 256", o, d.H);
        if (d.I < ci.bn / 2 || d.I % (ci.bn / 2) != 0 || d.I % (2 * ci.bk) != 0 || d.I % 256 != 0)
            return fail(MOE_ERR_UNSUPPORTED, "op %d: I=%d must be a positive multiple of 256", o, d.I);
        if (is_fp8_cls(cls)) {
            if (d.H > 128 * ShapeF8::MAX_KB || d.I > 128 * ShapeF8::MAX_KB)
                return fail(MOE_ERR_UNSUPPORTED, "op %d: fp8 H, I must be at most %d", o, 128 * ShapeF8::MAX_KB);
            if (!(d.x ? d.x_scales : d.x_perm_scales) || !d.w_gate_up_scales || !d.w_down_scales || !d.h_scales)
                return fail(MOE_ERR_INVALID_ARG, "op %d: fp8 op without its scale buffers", o);
        }
        if (d.row_align != kSegAlign)
            return fail(MOE_ERR_INVALID_ARG, "op %d: row_align=%d but the FFN needs segments aligned to %d rows", o,
                        d.row_align, kSegAlign);
        if (d.capacity < d.row_align) return fail(MOE_ERR_CAPACITY, "op %d: capacity=%d below one block", o, d.capacity);
        if ((int64_t)d.capacity * d.H > INT32_MAX || (int64_t)d.capacity * d.I > INT32_MAX)
            return fail(MOE_ERR_UNSUPPORTED, "op %d: capacity*H exceeds 2^31 elements", o);
        if (d.capacity / d.row_align >= kMaxRowTiles)
            return fail(MOE_ERR_UNSUPPORTED, "op %d: capacity=%d exceeds %d row tiles", o, d.capacity, kMaxRowTiles);
        if (!d.counts || !d.offsets || !d.w_gate_up || !d.w_down || !d.h || !d.y_perm)
            return fail(MOE_ERR_INVALID_ARG, "op %d: null buffer", o);
        // GEMM-1 operand: x_perm, or x gathered through row_to_assign (exactly one of the two)
        if ((d.x_perm != nullptr) == (d.x != nullptr))
            return fail(MOE_ERR_INVALID_ARG, "op %d: give exactly one of x_perm and x", o);
        if (d.x) {
            if (!d.row_to_assign || d.T < 1 || d.top_k < 1)
                return fail(MOE_ERR_INVALID_ARG, "op %d: gathered operand needs row_to_assign, T >= 1, top_k >= 1", o);
            if ((int64_t)d.T * d.H * (is_fp8_cls(cls) ? 1 : 2) >= ((int64_t)1 << 31))
                return fail(MOE_ERR_UNSUPPORTED, "op %d: T*H of the gathered operand exceeds 2^31 bytes", o);
        }
        if (d.y) {                                    // fused combine
            if (!d.assign_to_row || !d.topk_w || d.T < 0 || d.top_k < 1 || d.top_k > 32)
                return fail(MOE_ERR_INVALID_ARG, "op %d: fused combine needs assign_to_row, topk_w, T >= 0, top_k in [1,32]", o);
            if (d.y_dtype != MOE_BF16 && d.y_dtype != MOE_F32)
                return fail(MOE_ERR_UNSUPPORTED, "op %d: fused combine y_dtype %d not supported", o, d.y_dtype);
            if ((int64_t)d.T * d.top_k > INT32_MAX / 2 || (int64_t)d.T * d.H > INT32_MAX)
                return fail(MOE_ERR_UNSUPPORTED, "op %d: fused combine T too large", o);
        }
        if (d.depends_on_op >= o || d.depends_on_op < -1)
            return fail(MOE_ERR_INVALID_ARG, "op %d: depends_on_op=%d must be -1 or an earlier op", o, d.depends_on_op);
        if (d.gap_ns < 0) return fail(MOE_ERR_INVALID_ARG, "op %d: gap_ns < 0", o);
        OpArg& p = a.op[o];
        p.counts = d.counts;
        p.offsets = d.offsets;
        p.x = (const uint16_t*)(d.x ? d.x : d.x_perm);
        p.wgu = (const uint16_t*)d.w_gate_up;
        p.wd = (const uint16_t*)d.w_down;
        p.h = (uint16_t*)d.h;
        p.y = (uint16_t*)d.y_perm;
        p.xs = d.x ? d.x_scales : d.x_perm_scales;
        p.rmap = d.x ? d.row_to_assign : nullptr;
        p.T = d.x ? d.T : 0;
        p.top_k = d.x ? d.top_k : 1;
        p.wgus = d.w_gate_up_scales;
        p.wds = d.w_down_scales;
        p.hs = d.h_scales;
        p.done_word = d.done_word;
        p.a2r = d.y ? d.assign_to_row : nullptr;
        p.tw = d.y ? d.topk_w : nullptr;
        p.yc = d.y;
        p.ct = d.y ? d.T : 0;
        p.ck = d.y ? d.top_k : 1;
        p.y_f32 = d.y && d.y_dtype == MOE_F32;
        p.n3 = d.y ? (d.T + kCombTokens - 1) / kCombTokens : 0;
        p.cls = cls;
        p.phase = d.phase;
        p.layer = d.layer;
        p.E = d.E_local;
        p.H = d.H;
        p.I = d.I;
        p.capacity = d.capacity;
        p.mt = ci.bm;
        p.n1 = d.I / (ci.bn / 2);
        p.n2 = d.H / ci.bn;
        p.max_mtiles = (d.capacity + kSegAlign - 1) / kSegAlign + 1;   // row tiles never outnumber 32-row blocks
        size_t tb = 0, gb = 0;
        const size_t ob = op_array_bytes(d.capacity, kSegAlign, &tb, &gb);
        p.table_off = (int32_t)off;
        p.g1_off = (int32_t)(off + tb);
        p.grp_off = (int32_t)(off + tb + gb);
        p.qtab_off = (int32_t)(off + tb + 2 * gb);
        p.rel = d.release_word != nullptr;
        off += ob;
        ia.rel_words[o] = d.release_word;
        ia.rel_after[o] = d.release_after_ns < 0 ? -1 : d.release_after_ns * (int64_t)wc_khz / 1000000;
        ia.gaps[o] = d.gap_ns * (int64_t)wc_khz / 1000000;
        ia.deps[o] = d.depends_on_op;
        ia.phases[o] = d.phase;
    }
    return MOE_OK;
}

// The one launch path of both FFN entry points: checks, kernel arguments,
// the init kernel (which zeroes the scheduler state with ordinary stores) and
// the persistent kernel.  `workspace` holds at least ws_bytes_for(ops) bytes.
moe_status_t launch_ffn(const moe_op_desc* ops, int32_t n_ops, const moe_sched_config* cfg, void* workspace,
                        int32_t* status_word, void* stream) {
    using moeapk_host::fail;
    if (!ops || !cfg || !workspace || !status_word) return fail(MOE_ERR_INVALID_ARG, "moe_grouped_ffn_persistent: null pointer");
    if (n_ops < 1 || n_ops > MOE_MAX_OPS)
        return fail(MOE_ERR_INVALID_ARG, "moe_grouped_ffn_persistent: n_ops=%d outside [1,%d]", n_ops, MOE_MAX_OPS);
    int cu = 0, wc_khz = 0;
    moe_status_t st = moeapk_host::check_device(&cu, &wc_khz);
    if (st != MOE_OK) return st;

    KArgs a;
    memset(&a, 0, sizeof(a));
    InitArgs ia;
    memset(&ia, 0, sizeof(ia));
    size_t off = 0;
    if (cfg->prefill_tile_rows != 0 && cfg->prefill_tile_rows != 192 && cfg->prefill_tile_rows != 128)
        return fail(MOE_ERR_INVALID_ARG, "prefill_tile_rows=%d must be 0, 192 or 128", cfg->prefill_tile_rows);
    st = fill_ops(ops, n_ops, wc_khz, a, ia, off, cfg->prefill_tile_rows);
    if (st != MOE_OK) return st;
    if (kArraysOff + off > (size_t)INT32_MAX) return fail(MOE_ERR_UNSUPPORTED, "scheduler workspace too large");
    int n_wg = cfg->n_workgroups > 0 ? cfg->n_workgroups : cu;
    a.n_ops = n_ops;
    a.q = cfg->decode_quota_wg < 0 ? 0 : cfg->decode_quota_wg;
    a.q_max = cfg->decode_quota_max_wg > 0 ? cfg->decode_quota_max_wg : n_wg / 2;
    a.x_star = cfg->x_moe_expected;
    a.c = cfg->round_multiple > 0 ? cfg->round_multiple : 8;
    if (cfg->group_row_tiles < 0 || cfg->group_row_tiles > kMaxGroup)
        return fail(MOE_ERR_INVALID_ARG, "group_row_tiles=%d outside [0,%d]", cfg->group_row_tiles, kMaxGroup);
    a.gmax = cfg->group_row_tiles > 0 ? cfg->group_row_tiles : kDefaultGroup;
    // prefill tiles may be claimed ahead only by workgroups that no decode
    // quota can reach: q' <= Q_max, and with a fixed quota q' is known
    bool any_decode = false, any_prefill = false;
    for (int o = 0; o < n_ops; ++o) {
        any_decode |= ops[o].phase == MOE_DECODE;
        any_prefill |= ops[o].phase == MOE_PREFILL;
    }
    a.pre_dec_all = any_prefill ? 0 : 1;
    if (cfg->static_partition < 0 || cfg->static_partition > 1)
        return fail(MOE_ERR_INVALID_ARG, "static_partition=%d must be 0 or 1", cfg->static_partition);
    a.split = cfg->static_partition;
    if (a.split) {                                   // the split is the fixed q' (Eq. 4 with x*_moe <= 0)
        a.pre_wg = moeapk::decode_quota(a.q, 0, 0, a.q_max, a.c);
        a.pre_dec_all = 0;
        if (a.x_star > 0 || a.pre_wg < 1 || a.pre_wg >= n_wg)
            return fail(MOE_ERR_INVALID_ARG, "static_partition needs a fixed quota 0 < q' < n_workgroups");
    }
    a.pre_wg = !any_decode ? 0 : (a.x_star <= 0 ? moeapk::decode_quota(a.q, 0, 0, a.q_max, a.c) : a.q_max);
    // the smallest q' of any decode op (Eq. (4) is non-decreasing in x_moe >= 1)
    a.inst_wg = a.x_star <= 0 ? a.pre_wg : moeapk::decode_quota(a.q, 1, a.x_star, a.q_max, a.c);
    a.spin_limit = cfg->spin_limit > 0 ? cfg->spin_limit : (int64_t)2000000;
    a.abort_word = cfg->abort_word;
    a.trace = cfg->trace;
    a.trace_per_wg = cfg->trace ? cfg->trace_capacity / n_wg : 0;
    if (cfg->trace && a.trace_per_wg < 1)
        return fail(MOE_ERR_INVALID_ARG, "trace_capacity=%lld holds no record per workgroup (%d workgroups)",
                    (long long)cfg->trace_capacity, n_wg);
    a.stats = cfg->op_stats;
    a.status = status_word;
    a.ws = (char*)workspace;

    bool comb = false;
    for (int o = 0; o < n_ops; ++o) comb |= a.op[o].n3 > 0;
    const void* kfn = comb ? (const void*)apk_kernel<true> : (const void*)apk_kernel<false>;
    static bool attr_set[2] = {false, false};
    if (!attr_set[comb]) {
        if (hipFuncSetAttribute(kfn, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes) != hipSuccess)
            return fail(MOE_ERR_HIP, "hipFuncSetAttribute(LDS=%d) failed", kLdsBytes);
        attr_set[comb] = true;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kfn, 256, kLdsBytes) != hipSuccess)
        return fail(MOE_ERR_HIP, "occupancy query failed");
    if (per_cu < 1) return fail(MOE_ERR_UNSUPPORTED, "persistent kernel does not fit on a CU");
    if (n_wg > per_cu * cu) return fail(MOE_ERR_INVALID_ARG, "n_workgroups=%d exceeds co-resident capacity %d", n_wg, per_cu * cu);

    ia.n_ops = n_ops;
    ia.ws_vec = (int32_t)((kArraysOff + off) / 16);
    ia.ws = (char*)workspace;
    ia.status = status_word;
    hipStream_t s = (hipStream_t)stream;
    const int arr_vec = ia.ws_vec - (int)(kArraysOff / 16);
    const int init_wg = 1 + (arr_vec <= 0 ? 0 : (arr_vec + 1023) / 1024 < 16 ? (arr_vec + 1023) / 1024 : 16);
    hipLaunchKernelGGL(apk_init_kernel, dim3(init_wg), dim3(256), 0, s, ia);
    if (comb) hipLaunchKernelGGL(apk_kernel<true>, dim3(n_wg), dim3(256), kLdsBytes, s, a);
    else hipLaunchKernelGGL(apk_kernel<false>, dim3(n_wg), dim3(256), kLdsBytes, s, a);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_grouped_ffn_persistent: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}

// Static scheduler workspace of the allocation-free entry point, one copy per
// GPU (held until the process ends).  Host code never passes `scratch` itself
// to a kernel (in host code it names a host-side stand-in): its device address
// is taken once per device with hipGetSymbolAddress, with that device current.
static __device__ __align__(256) char scratch[MOE_FFN_NOALLOC_WORKSPACE_BYTES];
constexpr int kMaxScratchDevices = 64;
void* g_scratch_ptr[kMaxScratchDevices];
std::mutex g_scratch_mu;

moe_status_t scratch_address(void** ptr) {
    using moeapk_host::fail;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return fail(MOE_ERR_HIP, "hipGetDevice failed");
    if (dev < 0 || dev >= kMaxScratchDevices) return fail(MOE_ERR_UNSUPPORTED, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(MOE_ERR_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev, hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return MOE_OK;
}

// ----------------------------------------------------------------------------- plain-grid baseline
// The same tiles with no device scheduler: per op, a planning kernel builds the
// row-tile table (one workgroup), then one grid per GEMM runs its tiles round
// robin over one workgroup per CU, column block major so that consecutive
// workgroups share a weight slice; the kernel boundary is the GEMM-1 -> GEMM-2
// dependency.  For measuring what the persistent scheduler costs or saves.
struct PlainArgs {
    OpArg op;
    char* ws;
    int32_t o, gmax, reset_status;
    int32_t* status;
};

__global__ __launch_bounds__(256) void plain_plan_kernel(const PlainArgs p) {
    __shared__ int32_t scan[1024], s_cnt[1024], s_off[1024];
    __shared__ int32_t s_total, s_bad;
    if (p.reset_status && threadIdx.x == 0) *p.status = MOE_OK;
    __syncthreads();
    build_row_tiles(p.op, (uint64_t*)(arr_of(p.ws) + p.op.table_off), (uint32_t*)(arr_of(p.ws) + p.op.grp_off),
                    p.gmax, scan, s_cnt, s_off, &s_total, &s_bad);
    __syncthreads();
    if (threadIdx.x == 0) {
        if (s_bad) set_status(p.status, MOE_ERR_CAPACITY);
        dyn_of(p.ws)[p.o].x_moe = s_bad ? 0 : s_total;
    }
}

template <int STAGE>
__global__ __launch_bounds__(256, 1) void plain_gemm_kernel(const PlainArgs p) {
    extern __shared__ __align__(16) char lds[];
    const OpArg& op = p.op;
    const int xm = __builtin_amdgcn_readfirstlane(*(volatile const int32_t*)&dyn_of(p.ws)[p.o].x_moe);
    const int n = STAGE == 1 ? op.n1 : op.n2;
    const uint64_t* table = (const uint64_t*)(arr_of(p.ws) + op.table_off);
    for (int t = blockIdx.x; t < xm * n; t += gridDim.x) {
        const int nb = t / xm, mtile = t - nb * xm;
        int e, mblk, rows, row0;
        sched::unpack_entry(table[mtile], e, mblk, rows, row0);
        e = __builtin_amdgcn_readfirstlane(e);
        rows = __builtin_amdgcn_readfirstlane(rows);
        row0 = __builtin_amdgcn_readfirstlane(row0);
        const int rows32 = (rows + 31) & ~31;
        if (e >= op.E || rows < 1 || rows > op.mt || row0 < 0 || (long)row0 + rows32 > (long)op.capacity) {
            if (threadIdx.x == 0) set_status(p.status, MOE_ERR_INTERNAL);
            return;
        }
        run_tile(op, STAGE, row0, rows32, nb, e, lds, NoHook{});
        wait_own_stores();
        __syncthreads();                                      // the next tile reuses the LDS
    }
}

}  // namespace

extern "C" moe_status_t moe_grouped_ffn_plain(const moe_op_desc* ops, int32_t n_ops, void* workspace,
                                              int32_t* status_word, void* stream) {
    using moeapk_host::fail;
    if (!ops || !workspace || !status_word) return fail(MOE_ERR_INVALID_ARG, "moe_grouped_ffn_plain: null pointer");
    if (n_ops < 1 || n_ops > MOE_MAX_OPS)
        return fail(MOE_ERR_INVALID_ARG, "moe_grouped_ffn_plain: n_ops=%d outside [1,%d]", n_ops, MOE_MAX_OPS);
    int cu = 0, wc_khz = 0;
    moe_status_t st = moeapk_host::check_device(&cu, &wc_khz);
    if (st != MOE_OK) return st;
    KArgs a;
    memset(&a, 0, sizeof(a));
    InitArgs ia;
    memset(&ia, 0, sizeof(ia));
    size_t off = 0;
    st = fill_ops(ops, n_ops, wc_khz, a, ia, off);
    if (st != MOE_OK) return st;
    static bool attr_set = false;
    if (!attr_set) {
        if (hipFuncSetAttribute((const void*)plain_gemm_kernel<1>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                kLdsBytes) != hipSuccess ||
            hipFuncSetAttribute((const void*)plain_gemm_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                kLdsBytes) != hipSuccess)
            return fail(MOE_ERR_HIP, "hipFuncSetAttribute(LDS=%d) failed", kLdsBytes);
        attr_set = true;
    }
    hipStream_t s = (hipStream_t)stream;
    for (int o = 0; o < n_ops; ++o) {
        PlainArgs p;
        memset(&p, 0, sizeof(p));
        p.op = a.op[o];
        p.ws = (char*)workspace;
        p.o = o;
        p.gmax = kDefaultGroup;
        p.reset_status = o == 0;
        p.status = status_word;
        hipLaunchKernelGGL(plain_plan_kernel, dim3(1), dim3(256), 0, s, p);
        hipLaunchKernelGGL(plain_gemm_kernel<1>, dim3(cu), dim3(256), kLdsBytes, s, p);
        hipLaunchKernelGGL(plain_gemm_kernel<2>, dim3(cu), dim3(256), kLdsBytes, s, p);
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_grouped_ffn_plain: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}

extern "C" moe_status_t moe_grouped_ffn_persistent(const moe_op_desc* ops, int32_t n_ops, const moe_sched_config* cfg,
                                                   void* workspace, int32_t* status_word, void* stream) {
    return launch_ffn(ops, n_ops, cfg, workspace, status_word, stream);
}

extern "C" moe_status_t moe_grouped_ffn_persistent_noalloc(const moe_op_desc* ops, int32_t n_ops,
                                                           const moe_sched_config* cfg, int32_t* status_word,
                                                           void* stream) {
    using moeapk_host::fail;
    if (!ops || n_ops < 1 || n_ops > MOE_MAX_OPS)
        return fail(MOE_ERR_INVALID_ARG, "moe_grouped_ffn_persistent_noalloc: n_ops=%d outside [1,%d]", n_ops,
                    MOE_MAX_OPS);
    for (int o = 0; o < n_ops; ++o)
        if (ops[o].capacity < 0) return fail(MOE_ERR_INVALID_ARG, "op %d: capacity < 0", o);
    const size_t need = ws_bytes_for(ops, n_ops);
    if (need > (size_t)MOE_FFN_NOALLOC_WORKSPACE_BYTES)
        return fail(MOE_ERR_CAPACITY, "moe_grouped_ffn_persistent_noalloc: the ops need %zu bytes of scheduler "
                    "workspace, above the static %u", need, (unsigned)MOE_FFN_NOALLOC_WORKSPACE_BYTES);
    if (!cfg || !status_word) return fail(MOE_ERR_INVALID_ARG, "moe_grouped_ffn_persistent_noalloc: null pointer");
    moe_status_t st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    void* ws = nullptr;
    st = scratch_address(&ws);
    if (st != MOE_OK) return st;
    return launch_ffn(ops, n_ops, cfg, ws, status_word, stream);
}
