// a1: top-k softmax gating (Background, "MoE LLM Inference").
//
// One 64-wide wave per token.  Lane l holds experts l, l+64, ... as 32-bit
// order keys: the fp32 logit mapped to an unsigned integer that orders like the
// float (-0.0 folded onto +0.0; key 0 is kept for absent or retired experts).
// Each of the k rounds takes the wave-wide maximum key with DPP max steps
// inside each 16-lane row and four lane reads across the rows, then one ballot
// per lane slot finds the experts holding that key: the lowest such expert
// index wins (ties go to the lower index), is retired, and lane j keeps the
// winner of round j.  Rounds are bound by vector-ALU issue (four cycles per
// wave64 instruction), so keys stay 32 bits wide and the tie break is scalar.
#include <cstring>

#include "common.hpp"

namespace {

using moeapk::set_status;

constexpr int kTokensPerBlock = 4;  // one wave each

__device__ __forceinline__ uint32_t order_key(float v) {
    uint32_t u = __float_as_uint(v);
    if (u == 0x80000000u) u = 0u;                        // -0.0 ties with +0.0
    const uint32_t k = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return k > 1u ? k : 1u;                              // only a NaN pattern maps below 1
}

__device__ __forceinline__ float key_value(uint32_t k) {
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// DPP controls: quad permutes [1,0,3,2] and [2,3,0,1], half-row and row mirrors.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

// (0, the identity of an unsigned max, fills disabled lanes: the move folds into the max)
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_max(uint32_t v) {
    const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
    return v > o ? v : o;
}

// Maximum of v over the wave, the same value in every lane.
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
    v = dpp_max<kDppXor1>(v);
    v = dpp_max<kDppXor2>(v);
    v = dpp_max<kDppHalfMirror>(v);
    v = dpp_max<kDppMirror>(v);                          // every lane: its row's maximum
    const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
    const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
    const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
    const uint32_t a = r0 > r1 ? r0 : r1, b = r2 > r3 ? r2 : r3;
    return a > b ? a : b;
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_min(uint32_t v) {
    const uint32_t o = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, false);
    return v < o ? v : o;
}

// Minimum of v over the wave, the same value in every lane.
__device__ __forceinline__ uint32_t wave_min(uint32_t v) {
    v = dpp_min<kDppXor1>(v);
    v = dpp_min<kDppXor2>(v);
    v = dpp_min<kDppHalfMirror>(v);
    v = dpp_min<kDppMirror>(v);
    const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
    const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
    const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
    const uint32_t a = r0 < r1 ? r0 : r1, b = r2 < r3 ? r2 : r3;
    return a < b ? a : b;
}

// (key, expert) pairs in selection order: larger key first, then lower expert.
__device__ __forceinline__ void order_pair(uint32_t& ka, uint32_t& ia, uint32_t& kb, uint32_t& ib) {
    const bool swap = kb > ka || (kb == ka && ib < ia);
    const uint32_t k0 = swap ? kb : ka, i0 = swap ? ib : ia;
    kb = swap ? ka : kb;
    ib = swap ? ia : ib;
    ka = k0;
    ia = i0;
}

// Sum of v over the wave, the same value in every lane.
__device__ __forceinline__ float wave_sum(float v) {
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kDppXor1, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kDppXor2, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kDppHalfMirror, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kDppMirror, 0xF, 0xF, false));
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

// One wave's token t: writes its ids and weights and returns, in lanes
// j < k, the local expert of slot j (-1 if not local; -1 in every lane when
// t >= T, which writes nothing).
template <int EPL>
__device__ __forceinline__ int route_wave(const float* __restrict__ logits, int t, int T, int E, int k,
                                          int local_begin, int E_local, int32_t* __restrict__ ids,
                                          float* __restrict__ wts) {
    const int lane = threadIdx.x & 63;
    if (t >= T) return -1;  // wave-uniform
    const float* row = logits + (size_t)t * E;
    // all loads first (clamped in-row indices, no branches), so they are in flight together
    float v[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) v[i] = row[min(lane + 64 * i, E - 1)];
    uint32_t key[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) key[i] = (lane + 64 * i < E) ? order_key(v[i]) : 0u;
    int my_e = -1;
    uint32_t my_key = 0;
    if constexpr (EPL <= 4) {
        // Each lane sorts its pairs once; a round then reduces only the lanes'
        // heads, and the lane holding the winner drops its head.  The winner is
        // the largest key, ties to the lower expert: a unique maximum head is
        // found with one ballot; equal heads in several lanes take a wave-wide
        // minimum over their experts.
        uint32_t idx[EPL];
#pragma unroll
        for (int i = 0; i < EPL; ++i) idx[i] = (uint32_t)(lane + 64 * i);
        if constexpr (EPL >= 2) order_pair(key[0], idx[0], key[1], idx[1]);
        if constexpr (EPL == 4) {
            order_pair(key[2], idx[2], key[3], idx[3]);
            order_pair(key[0], idx[0], key[2], idx[2]);
            order_pair(key[1], idx[1], key[3], idx[3]);
            order_pair(key[1], idx[1], key[2], idx[2]);
        }
        for (int r = 0; r < k; ++r) {
            const uint32_t best = wave_max(key[0]);
            const uint64_t hit = __ballot(key[0] == best);
            int e;
            if (__popcll(hit) == 1) e = __builtin_amdgcn_readlane((int)idx[0], __ffsll((long long)hit) - 1);
            else e = (int)wave_min(key[0] == best ? idx[0] : 0xFFFFFFFFu);
            if (lane == (e & 63)) {                          // drop the winner from its lane
#pragma unroll
                for (int i = 0; i + 1 < EPL; ++i) { key[i] = key[i + 1]; idx[i] = idx[i + 1]; }
                key[EPL - 1] = 0u;
            }
            if (lane == r) {
                my_e = e;
                my_key = best;
            }
        }
    } else {
    for (int r = 0; r < k; ++r) {
        uint32_t best = key[0];
#pragma unroll
        for (int i = 1; i < EPL; ++i) best = key[i] > best ? key[i] : best;
        best = wave_max(best);
        // lowest expert index holding the maximum: the first slot with a hit, its lowest lane
        int e = 0;
#pragma unroll
        for (int i = EPL - 1; i >= 0; --i) {
            const uint64_t hit = __ballot(key[i] == best);
            if (hit) e = 64 * i + __ffsll((long long)hit) - 1;
        }
        const int wl = e & 63, wi = e >> 6;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
            if (i == wi && lane == wl) key[i] = 0u;      // retire the winner
        if (lane == r) {
            my_e = e;
            my_key = best;
        }
    }
    }
    const int loc = my_e - local_begin;
    const bool local = lane < k && loc >= 0 && loc < E_local;
    const float my_v = key_value(my_key);
    const float m = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_v), 0));   // the largest selected logit
    const float ex = (lane < k) ? expf(my_v - m) : 0.f;
    const float s = wave_sum(ex);
    if (lane < k) {
        ids[(size_t)t * k + lane] = local ? loc : -1;
        wts[(size_t)t * k + lane] = ex / s;
    }
    return local ? loc : -1;
}

// Unmasked routing: block `blk` of the op handles tokens [4*blk, 4*blk + 4).
template <int EPL>
__device__ __forceinline__ void route_block(const float* __restrict__ logits, int T, int E, int k, int local_begin,
                                            int E_local, int32_t* __restrict__ ids, float* __restrict__ wts,
                                            int blk) {
    route_wave<EPL>(logits, blk * kTokensPerBlock + (threadIdx.x >> 6), T, E, k, local_begin, E_local, ids, wts);
}

// ----------------------------------------------------------------------------- masked placement
// Masked layout ("Prefill-Decode Disaggregation": a fixed region of `slots`
// rows per local expert and a count, filled as routing decides): slot
// a = t*k + j of local expert e goes to row e*slots + (number of earlier
// assignments of e), so the rows of a region are its assignments in
// ascending a -- the unique order the permutation uses, bit-exact and
// independent of scheduling.
//
// A routing block of a masked op takes its chunk of 4 or 16 tokens from an ordered
// ticket (so every chunk it waits for belongs to a block that has already
// started), ranks its slots inside the chunk, publishes the chunk's
// per-expert counts and finds the counts of all earlier chunks by a
// decoupled look-back: walking back over the earlier chunks' records, summing
// aggregates until one holds an inclusive prefix.  Each record is one 64-bit
// word [generation | status | count], read and written with device-scope
// atomics, so no fence is needed; the generation (taken with the ticket from
// one word) makes records of earlier calls invalid without clearing them.
// The block that draws the last ticket resets the ticket and advances the
// generation; it also writes the counts (the inclusive prefix of the last
// chunk).
constexpr uint64_t kRecAgg = 1ull << 30, kRecIncl = 2ull << 30;
constexpr uint32_t kRecCountMask = (1u << 30) - 1;
constexpr int kPlaceHdrWords = 32;          // 256-byte header: the ticket word, alone in its line
// Tokens per masked block: one per wave up to kMaskedSmallT tokens (the
// block's latency is one token's routing), four per wave above (a quarter of
// the tickets on the op's ordered counter).
constexpr int kMaskedChunk = 16;
constexpr int kMaskedSmallT = 2048;
__host__ __device__ __forceinline__ int masked_chunk(int T) { return T <= kMaskedSmallT ? 4 : kMaskedChunk; }
constexpr int kMaskedMaxE = 1024;
constexpr int64_t kLookbackSpins = 1 << 22;

__device__ __forceinline__ uint64_t rec_word(uint32_t gen, uint64_t status, uint32_t count) {
    return ((uint64_t)gen << 32) | status | (uint64_t)(count & kRecCountMask);
}

struct MaskedArgs {
    int32_t* counts;
    int32_t* a2r;
    int32_t* r2a;
    uint64_t* ws;
    int32_t* err;
    int slots, nchunks;
};

template <int EPL, int CPW>
__device__ void route_block_masked(const float* __restrict__ logits, int T, int E, int k, int local_begin,
                                   int E_local, int32_t* __restrict__ ids, float* __restrict__ wts,
                                   const MaskedArgs m) {
    __shared__ int s_chunk;
    __shared__ uint32_t s_gen;
    __shared__ int32_t s_sel[kMaskedChunk][32];
    __shared__ int32_t s_cnt[kMaskedMaxE];
    __shared__ int32_t s_excl[kMaskedMaxE];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    if (tid == 0) {
        const unsigned long long old = atomicAdd((unsigned long long*)m.ws, 1ull);
        int c = (int)(uint32_t)old;
        const uint32_t gen = (uint32_t)(old >> 32);
        // the last ticket of the call: every other block has drawn its ticket already
        if (c == m.nchunks - 1)
            __hip_atomic_store(m.ws, (uint64_t)(gen + 1u) << 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (c >= m.nchunks) {                     // the workspace was not zero before its first use
            set_status(m.err, MOE_ERR_INTERNAL);
            c = -1;
        }
        s_chunk = c;
        s_gen = gen;
    }
    for (int e = tid; e < E_local; e += 256) s_cnt[e] = 0;
    __syncthreads();
    const int chunk = s_chunk;
    if (chunk < 0) return;                        // block-uniform
    const uint32_t gen = s_gen;
    // wave w routes tokens w, w + 4, ... of the chunk (chunk-local index tl = 4*it + w)
    int loc[CPW];
#pragma unroll
    for (int it = 0; it < CPW; ++it) {
        const int tl = it * kTokensPerBlock + w;
        loc[it] = route_wave<EPL>(logits, chunk * CPW * kTokensPerBlock + tl, T, E, k, local_begin, E_local, ids,
                                  wts);
        if (lane < 32) s_sel[tl][lane] = lane < k ? loc[it] : -1;
        if (loc[it] >= 0) atomicAdd(&s_cnt[loc[it]], 1);
    }
    __syncthreads();
    uint64_t* rec = m.ws + kPlaceHdrWords + (size_t)chunk * E_local;
    // publish first (chunk 0 holds its own inclusive prefix), then look back:
    // a block waits only on the records of earlier chunks, so no wait is circular
    for (int e = tid; e < E_local; e += 256)
        __hip_atomic_store(rec + e, rec_word(gen, chunk == 0 ? kRecIncl : kRecAgg, (uint32_t)s_cnt[e]),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int e = tid; e < E_local; e += 256) {
        uint32_t excl = 0;
        int64_t spins = 0;
        for (int j = chunk - 1; j >= 0;) {
            const uint64_t v = __hip_atomic_load(m.ws + kPlaceHdrWords + (size_t)j * E_local + e, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
            const uint64_t st = v & (3ull << 30);
            if ((uint32_t)(v >> 32) != gen || st == 0) {         // chunk j has not published yet
                if (++spins > kLookbackSpins) {
                    set_status(m.err, MOE_ERR_TIMEOUT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
                continue;
            }
            excl += (uint32_t)v & kRecCountMask;
            if (st == kRecIncl) break;
            --j;
        }
        if (chunk > 0)
            __hip_atomic_store(rec + e, rec_word(gen, kRecIncl, excl + (uint32_t)s_cnt[e]), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        s_excl[e] = (int32_t)excl;
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < CPW; ++it) {
        const int tl = it * kTokensPerBlock + w;
        const int t = chunk * CPW * kTokensPerBlock + tl;
        if (t >= T || lane >= k) continue;
        const int a = t * k + lane;
        int row = -1;
        if (loc[it] >= 0) {
            // rank inside the chunk: the chunk's earlier tokens that chose the same expert
            int r = s_excl[loc[it]];
            for (int t2 = 0; t2 < tl; ++t2)
                for (int j = 0; j < k; ++j) r += s_sel[t2][j] == loc[it];
            if (r < m.slots) {                    // always, as slots >= T
                row = loc[it] * m.slots + r;
                m.r2a[row] = a;
            } else {
                set_status(m.err, MOE_ERR_CAPACITY);
            }
        }
        m.a2r[a] = row;
    }
    if (chunk == m.nchunks - 1)
        for (int e = tid; e < E_local; e += 256) m.counts[e] = s_excl[e] + s_cnt[e];
}

template <int EPL>
__global__ __launch_bounds__(256) void topk_route_kernel(const float* __restrict__ logits, int T, int E, int k,
                                                        int local_begin, int E_local, int32_t* __restrict__ ids,
                                                        float* __restrict__ wts) {
    route_block<EPL>(logits, T, E, k, local_begin, E_local, ids, wts, blockIdx.x);
}

// Several ops in one launch: entry o owns blocks [blk0[o], blk0[o + 1]); the
// host puts masked entries first, so their longer blocks are dispatched first.
struct RouteBatch {
    moe_route_args op[MOE_MAX_OPS];
    int32_t blk0[MOE_MAX_OPS + 1];
    int32_t n;
};

template <int EPL>
__global__ __launch_bounds__(256) void topk_route_batch_kernel(const RouteBatch b) {
    int o = 0;
    while (o + 1 < b.n && (int)blockIdx.x >= b.blk0[o + 1]) ++o;      // uniform
    const moe_route_args& a = b.op[o];
    if (a.counts) {
        const MaskedArgs m{a.counts, a.assign_to_row, a.row_to_assign, (uint64_t*)a.place_ws, a.error_flag, a.slots,
                           b.blk0[o + 1] - b.blk0[o]};
        if (masked_chunk(a.T) == 4)
            route_block_masked<EPL, 1>(a.logits, a.T, a.E_global, a.top_k, a.local_begin, a.E_local, a.topk_ids,
                                       a.topk_w, m);
        else
            route_block_masked<EPL, kMaskedChunk / kTokensPerBlock>(a.logits, a.T, a.E_global, a.top_k,
                                                                     a.local_begin, a.E_local, a.topk_ids, a.topk_w, m);
        return;
    }
    route_block<EPL>(a.logits, a.T, a.E_global, a.top_k, a.local_begin, a.E_local, a.topk_ids, a.topk_w,
                     (int)blockIdx.x - b.blk0[o]);
}

moe_status_t check_route(const float* logits, int32_t T, int32_t E_global, int32_t top_k, int32_t local_begin,
                         int32_t E_local, const int32_t* topk_ids, const float* topk_w) {
    using moeapk_host::fail;
    if (T < 0) return fail(MOE_ERR_INVALID_ARG, "moe_topk_route: T=%d < 0", T);
    if (E_global < 1 || E_global > 1024)
        return fail(MOE_ERR_UNSUPPORTED, "moe_topk_route: E_global=%d outside [1,1024]", E_global);
    if (top_k < 1 || top_k > E_global || top_k > 32)
        return fail(MOE_ERR_INVALID_ARG, "moe_topk_route: top_k=%d outside [1, min(E_global,32)]", top_k);
    if (local_begin < 0 || E_local < 1)
        return fail(MOE_ERR_INVALID_ARG, "moe_topk_route: local_begin=%d E_local=%d", local_begin, E_local);
    if (T > 0 && (!logits || !topk_ids || !topk_w)) return fail(MOE_ERR_INVALID_ARG, "moe_topk_route: null pointer");
    return MOE_OK;
}

}  // namespace

extern "C" moe_status_t moe_topk_route(const float* logits, int32_t T, int32_t E_global, int32_t top_k,
                                       int32_t local_begin, int32_t E_local, int32_t* topk_ids, float* topk_w,
                                       void* stream) {
    using moeapk_host::fail;
    moe_status_t st = check_route(logits, T, E_global, top_k, local_begin, E_local, topk_ids, topk_w);
    if (st != MOE_OK) return st;
    if (T == 0) return MOE_OK;
    st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid((T + kTokensPerBlock - 1) / kTokensPerBlock), block(256);
    const int epl = (E_global + 63) / 64;
    if (epl <= 1) hipLaunchKernelGGL(topk_route_kernel<1>, grid, block, 0, s, logits, T, E_global, top_k, local_begin, E_local, topk_ids, topk_w);
    else if (epl <= 2) hipLaunchKernelGGL(topk_route_kernel<2>, grid, block, 0, s, logits, T, E_global, top_k, local_begin, E_local, topk_ids, topk_w);
    else if (epl <= 4) hipLaunchKernelGGL(topk_route_kernel<4>, grid, block, 0, s, logits, T, E_global, top_k, local_begin, E_local, topk_ids, topk_w);
    else if (epl <= 8) hipLaunchKernelGGL(topk_route_kernel<8>, grid, block, 0, s, logits, T, E_global, top_k, local_begin, E_local, topk_ids, topk_w);
    else hipLaunchKernelGGL(topk_route_kernel<16>, grid, block, 0, s, logits, T, E_global, top_k, local_begin, E_local, topk_ids, topk_w);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_topk_route: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}

extern "C" size_t moe_route_place_workspace_bytes(int32_t T, int32_t E_local) {
    if (T < 1 || E_local < 1) return 0;
    // the most chunks of any call with up to T tokens (4-token chunks reach
    // kMaskedSmallT / 4 of them before the chunk grows to 16 tokens)
    size_t chunks = (size_t)((T + masked_chunk(T) - 1) / masked_chunk(T));
    if (T > kMaskedSmallT && chunks < (size_t)(kMaskedSmallT / 4)) chunks = kMaskedSmallT / 4;
    return (kPlaceHdrWords + chunks * (size_t)E_local) * sizeof(uint64_t);
}

extern "C" moe_status_t moe_topk_route_batch(const moe_route_args* ops, int32_t n_ops, void* stream) {
    using moeapk_host::fail;
    if (!ops || n_ops < 1 || n_ops > MOE_MAX_OPS)
        return fail(MOE_ERR_INVALID_ARG, "moe_topk_route_batch: n_ops=%d outside [1,%d]", n_ops, MOE_MAX_OPS);
    RouteBatch b;
    memset(&b, 0, sizeof(b));
    int epl = 1;
    int64_t blocks = 0;
    for (int o = 0; o < n_ops; ++o) {
        const moe_route_args& a = ops[o];
        const moe_status_t st = check_route(a.logits, a.T, a.E_global, a.top_k, a.local_begin, a.E_local,
                                            a.topk_ids, a.topk_w);
        if (st != MOE_OK) return st;
        if (a.counts) {
            if (a.T < 1 || a.slots < a.T || a.slots % 32 != 0 || (int64_t)a.slots * a.E_local > INT32_MAX ||
                a.T >= (1 << 29))
                return fail(MOE_ERR_INVALID_ARG, "moe_topk_route_batch: entry %d: masked layout needs 1 <= T < 2^29 and "
                            "slots (%d) a multiple of 32, >= T=%d, slots*E_local < 2^31", o, a.slots, a.T);
            if (a.E_local > kMaskedMaxE || a.top_k > 32)
                return fail(MOE_ERR_UNSUPPORTED, "moe_topk_route_batch: entry %d: masked layout needs E_local <= %d",
                            o, kMaskedMaxE);
            if (!a.assign_to_row || !a.row_to_assign || !a.place_ws)
                return fail(MOE_ERR_INVALID_ARG, "moe_topk_route_batch: entry %d: masked layout needs assign_to_row, "
                            "row_to_assign and place_ws", o);
            if ((uintptr_t)a.place_ws % 8 != 0)
                return fail(MOE_ERR_INVALID_ARG, "moe_topk_route_batch: entry %d: place_ws must be 8-byte aligned", o);
        }
        const int e = (a.E_global + 63) / 64;
        epl = e > epl ? e : epl;
    }
    int n = 0;
    for (int pass = 0; pass < 2; ++pass)                  // masked entries first, then the others
        for (int o = 0; o < n_ops; ++o) {
            const moe_route_args& a = ops[o];
            if ((a.counts != nullptr) != (pass == 0)) continue;
            b.op[n] = a;
            b.blk0[n] = (int32_t)blocks;
            const int per = a.counts ? masked_chunk(a.T) : kTokensPerBlock;
            blocks += (a.T + per - 1) / per;
            ++n;
        }
    if (blocks > INT32_MAX) return fail(MOE_ERR_UNSUPPORTED, "moe_topk_route_batch: too many tokens");
    b.blk0[n_ops] = (int32_t)blocks;
    b.n = n_ops;
    if (blocks == 0) return MOE_OK;
    moe_status_t st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid((unsigned)blocks), block(256);
    if (epl <= 1) hipLaunchKernelGGL(topk_route_batch_kernel<1>, grid, block, 0, s, b);
    else if (epl <= 2) hipLaunchKernelGGL(topk_route_batch_kernel<2>, grid, block, 0, s, b);
    else if (epl <= 4) hipLaunchKernelGGL(topk_route_batch_kernel<4>, grid, block, 0, s, b);
    else if (epl <= 8) hipLaunchKernelGGL(topk_route_batch_kernel<8>, grid, block, 0, s, b);
    else hipLaunchKernelGGL(topk_route_batch_kernel<16>, grid, block, 0, s, b);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_topk_route_batch: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}
