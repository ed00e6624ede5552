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

// One op's routing: block `blk` of the op handles tokens [4*blk, 4*blk + 4).
// Masked layout outputs of an op (counts NULL: none).
struct MaskedOut {
    int32_t* counts;
    int32_t* a2r;
    int32_t* r2a;
    int slots;
};

template <int EPL>
__device__ __forceinline__ void route_block(const float* __restrict__ logits, int T, int E, int k, int local_begin,
                                            int E_local, int32_t* __restrict__ ids, float* __restrict__ wts, int blk,
                                            MaskedOut mo = MaskedOut{nullptr, nullptr, nullptr, 0}) {
    const int lane = threadIdx.x & 63;
    const int t = blk * kTokensPerBlock + (threadIdx.x >> 6);
    if (t >= T) return;  // wave-uniform
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
    // masked layout: claim the slot's row now, so the atomic's round trip overlaps the softmax
    const int loc = my_e - local_begin;
    const bool local = lane < k && loc >= 0 && loc < E_local;
    int slot = 0;
    if (mo.counts && local) slot = atomicAdd(mo.counts + loc, 1);
    const float my_v = key_value(my_key);
    const float m = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_v), 0));   // the largest selected logit
    const float ex = (lane < k) ? expf(my_v - m) : 0.f;
    const float s = wave_sum(ex);
    if (lane < k) {
        ids[(size_t)t * k + lane] = local ? loc : -1;
        wts[(size_t)t * k + lane] = ex / s;
        if (mo.counts) {                                 // masked layout: the next free row of the expert's region
            const int a = t * k + lane;
            int row = -1;
            if (local && slot < mo.slots) {              // always, as slots >= T
                row = loc * mo.slots + slot;
                mo.r2a[row] = a;
            }
            mo.a2r[a] = row;
        }
    }
}

template <int EPL>
__global__ __launch_bounds__(256) void topk_route_kernel(const float* __restrict__ logits, int T, int E, int k,
                                                        int local_begin, int E_local, int32_t* __restrict__ ids,
                                                        float* __restrict__ wts) {
    route_block<EPL>(logits, T, E, k, local_begin, E_local, ids, wts, blockIdx.x);
}

// Several ops in one launch: op o owns blocks [blk0[o], blk0[o + 1]).
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
    if (a.clear && (int)blockIdx.x == b.blk0[o])
        for (int i = threadIdx.x; i < a.E_local; i += 256) a.clear[i] = 0;
    route_block<EPL>(a.logits, a.T, a.E_global, a.top_k, a.local_begin, a.E_local, a.topk_ids, a.topk_w,
                     (int)blockIdx.x - b.blk0[o], MaskedOut{a.counts, a.assign_to_row, a.row_to_assign, a.slots});
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
            if (a.slots < a.T || a.slots % 32 != 0 || (int64_t)a.slots * a.E_local > INT32_MAX)
                return fail(MOE_ERR_INVALID_ARG, "moe_topk_route_batch: entry %d: slots=%d must be a multiple of 32, "
                            ">= T=%d, slots*E_local < 2^31", o, a.slots, a.T);
            if (!a.assign_to_row || !a.row_to_assign || a.clear == a.counts)
                return fail(MOE_ERR_INVALID_ARG, "moe_topk_route_batch: entry %d: masked layout needs assign_to_row, "
                            "row_to_assign and a clear array other than counts", o);
        }
        if (a.T == 0 && a.clear) return fail(MOE_ERR_INVALID_ARG, "moe_topk_route_batch: entry %d: clear with T=0", o);
        b.op[o] = a;
        b.blk0[o] = (int32_t)blocks;
        blocks += (a.T + kTokensPerBlock - 1) / kTokensPerBlock;
        const int e = (a.E_global + 63) / 64;
        epl = e > epl ? e : epl;
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
