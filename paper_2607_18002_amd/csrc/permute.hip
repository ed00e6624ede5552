// a2: permutation into per-expert contiguous segments at final offsets
// (Background, "Prefill-Decode Disaggregation": contiguous layout;
// "One-Sided Dispatch and Combine": each expert's destination and final offset
// are fixed after routing, before the activations are written).
//
// Two launches on the caller's stream, three with the activation copy:
//   count   : per-chunk expert histogram in LDS (512 assignments per block);
//             the last block to finish (a ticket counter in the workspace)
//             runs the scan: expert counts, padded segment offsets and the
//             per-(chunk, expert) bases, each expert's prefix over chunks
//             split across 256/E threads
//   scatter : stable rank of every assignment inside its chunk, built from
//             wave ballots (rank = popcount(match & lanes-below)) plus per-wave
//             and per-iteration running counts -> row_to_assign / assign_to_row.
//             The result is the unique order "ascending assignment a = t*k+j",
//             so it is bit-exact and independent of scheduling.  The same
//             launch marks every padding row of the segments -1.
//   gather  : only with x_perm: one wave per row copies x[a / k] (16-byte
//             vectors) into x_perm and zero-fills padding rows.
#include <cstring>

#include "common.hpp"

namespace {

using moeapk::set_status;

constexpr int kThreads = 256;
constexpr int kIters = 2;
constexpr int kChunk = kThreads * kIters;   // assignments per block

// Exclusive prefix over the E padded segment sizes by one 256-thread block:
// each thread scans a run of up to 4 experts, the run totals are scanned in LDS.
__device__ void block_offsets(int E, int align, int capacity, const int32_t* tot, int32_t* padded_off,
                              int32_t* counts, int32_t* offsets, int32_t* err) {
    __shared__ int32_t run_sum[kThreads];
    const int t = threadIdx.x;
    const int per = (E + kThreads - 1) / kThreads;             // 1..4 experts per thread
    const int e0 = t * per, e1 = min(E, e0 + per);
    int sum = 0;
    for (int e = e0; e < e1; ++e) sum += ((tot[e] + align - 1) / align) * align;
    run_sum[t] = sum;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {             // inclusive Hillis-Steele scan of the runs
        const int v = (t >= off) ? run_sum[t - off] : 0;
        __syncthreads();
        run_sum[t] += v;
        __syncthreads();
    }
    int base = run_sum[t] - sum;
    for (int e = e0; e < e1; ++e) {
        counts[e] = tot[e];
        offsets[e] = base;
        padded_off[e] = base;
        base += ((tot[e] + align - 1) / align) * align;
    }
    if (t == kThreads - 1) {
        offsets[E] = run_sum[t];
        if (run_sum[t] > capacity) set_status(err, MOE_ERR_CAPACITY);
    }
    __syncthreads();
}

// Block blk (of NB) of one op's count pass.
__device__ __forceinline__ void count_block(const int32_t* __restrict__ ids, int A, int E, int NB, int align,
                                            int capacity, unsigned* __restrict__ ticket,
                                            int32_t* __restrict__ blk_cnt,   // counts, then bases
                                            int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
                                            int32_t* __restrict__ err, int blk) {
    extern __shared__ int32_t hist[];                          // [E] histogram, later [E] totals + [E] offsets
    __shared__ int32_t part[kThreads * 4];                     // per (expert, run): run sum, then run base
    __shared__ int s_last;
    for (int e = threadIdx.x; e < E; e += kThreads) hist[e] = 0;
    __syncthreads();
    const int base = blk * kChunk;
    for (int it = 0; it < kIters; ++it) {
        const int a = base + it * kThreads + threadIdx.x;
        if (a < A) {
            const int id = ids[a];
            if (id < -1 || id >= E) set_status(err, MOE_ERR_BAD_EXPERT);
            else if (id >= 0) atomicAdd(&hist[id], 1);
        }
    }
    __syncthreads();
    // Publish this block's counts, then take a ticket; the last block scans.
    // The counts go out as device-coherent stores and every wave waits for its
    // own before the barrier, so the ticket needs no fence: a device-scope fence
    // here would write back the whole L2 of the XCD once per block.  The last
    // block reads the counts with coherent loads for the same reason.
    // atomicInc wraps to 0 on the last ticket, so the counter is ready for the next call.
    for (int e = threadIdx.x; e < E; e += kThreads)
        __hip_atomic_store(blk_cnt + (size_t)blk * E + e, hist[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    moeapk::wait_own_stores();
    __syncthreads();
    if (threadIdx.x == 0) s_last = atomicInc(ticket, (unsigned)(NB - 1)) == (unsigned)(NB - 1);
    __syncthreads();
    if (!s_last) return;

    // Scan.  P threads per expert (the largest power of two with P*E <= 256, at
    // least 1); unit u = (e, j) sums chunks [j*R, (j+1)*R) of expert e.
    int P = 1;
    while (P * 2 * E <= kThreads) P *= 2;
    const int U = P * E;                                        // <= 1024
    const int R = (NB + P - 1) / P;
    for (int u = threadIdx.x; u < U; u += kThreads) {
        const int e = u / P, j = u - e * P;
        const int b0 = j * R, b1 = min(NB, b0 + R);
        int sum = 0;
        int b = b0;
        for (; b + 8 <= b1; b += 8) {                          // eight independent loads in flight
            int c[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) c[i] = moeapk::ld_relaxed_agent(blk_cnt + (size_t)(b + i) * E + e);
#pragma unroll
            for (int i = 0; i < 8; ++i) sum += c[i];
        }
        for (; b < b1; ++b) sum += moeapk::ld_relaxed_agent(blk_cnt + (size_t)b * E + e);
        part[u] = sum;
    }
    __syncthreads();
    int32_t* tot = hist;                                        // reuse: E totals
    int32_t* poff = hist + E;                                   // E padded offsets
    for (int e = threadIdx.x; e < E; e += kThreads) {           // exclusive prefix over the expert's P runs
        int run = 0;
        for (int q = 0; q < P; ++q) { const int v = part[e * P + q]; part[e * P + q] = run; run += v; }
        tot[e] = run;
    }
    __syncthreads();
    block_offsets(E, align, capacity, tot, poff, counts, offsets, err);
    for (int u = threadIdx.x; u < U; u += kThreads) {           // bases of the unit's chunks
        const int e = u / P, j = u - e * P;
        const int b0 = j * R, b1 = min(NB, b0 + R);
        int run = poff[e] + part[u];
        int b = b0;
        for (; b + 8 <= b1; b += 8) {
            int c[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) c[i] = moeapk::ld_relaxed_agent(blk_cnt + (size_t)(b + i) * E + e);
#pragma unroll
            for (int i = 0; i < 8; ++i) { blk_cnt[(size_t)(b + i) * E + e] = run; run += c[i]; }
        }
        for (; b < b1; ++b) {
            const int c = moeapk::ld_relaxed_agent(blk_cnt + (size_t)b * E + e);
            blk_cnt[(size_t)b * E + e] = run;
            run += c;
        }
    }
}

// Block blk (of NB) of one op's scatter pass.
__device__ __forceinline__ void scatter_block(const int32_t* __restrict__ ids, int A, int E, int capacity,
                                              const int32_t* __restrict__ blk_base,
                                              const int32_t* __restrict__ counts,
                                              const int32_t* __restrict__ offsets,
                                              int32_t* __restrict__ row_to_assign,
                                              int32_t* __restrict__ assign_to_row, int32_t* __restrict__ err,
                                              int blk, int NB) {
    // padding rows [offsets[e] + counts[e], offsets[e+1]) of experts e = blk, blk + NB, ...
    for (int e = blk; e < E; e += NB) {
        const int r0 = offsets[e] + counts[e], r1 = min(offsets[e + 1], capacity);
        for (int r = r0 + (int)threadIdx.x; r < r1; r += kThreads) row_to_assign[r] = -1;
    }
    extern __shared__ int32_t sm[];
    int32_t* running = sm;           // [E]   rows handed out in earlier iterations
    int32_t* wcnt = sm + E;          // [4][E] per-wave counts of the current iteration
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int i = tid; i < 5 * E; i += kThreads) sm[i] = 0;
    __syncthreads();
    const int base = blk * kChunk;
    const int32_t* my_base = blk_base + (size_t)blk * E;
    for (int it = 0; it < kIters; ++it) {
        const int a = base + it * kThreads + tid;
        int id = (a < A) ? ids[a] : -1;
        if (id < -1 || id >= E) id = -1;                      // reported by the count kernel
        int rank = 0;
        uint64_t todo = __ballot(id >= 0);
        while (todo) {                                        // one pass per distinct expert in the wave
            const int leader = __ffsll((long long)todo) - 1;
            const int e = __shfl(id, leader, 64);
            const uint64_t match = __ballot(id == e);
            if (id == e) rank = __popcll(match & __lanemask_lt());
            if (lane == leader) wcnt[wave * E + e] = __popcll(match);
            todo &= ~match;
        }
        __syncthreads();
        if (id >= 0) {
            int prior = running[id];
            for (int w = 0; w < wave; ++w) prior += wcnt[w * E + id];
            const int row = my_base[id] + prior + rank;
            if (row < capacity) {
                row_to_assign[row] = a;
                assign_to_row[a] = row;
            } else {
                set_status(err, MOE_ERR_CAPACITY);
                assign_to_row[a] = -1;
            }
        } else if (a < A) {
            assign_to_row[a] = -1;
        }
        __syncthreads();
        for (int e = tid; e < E; e += kThreads)
            running[e] += wcnt[e] + wcnt[E + e] + wcnt[2 * E + e] + wcnt[3 * E + e];
        __syncthreads();
        for (int i = tid; i < 4 * E; i += kThreads) wcnt[i] = 0;
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void permute_count_kernel(const int32_t* __restrict__ ids, int A, int E, int NB,
                                                           int align, int capacity, unsigned* __restrict__ ticket,
                                                           int32_t* __restrict__ blk_cnt, int32_t* __restrict__ counts,
                                                           int32_t* __restrict__ offsets, int32_t* __restrict__ err) {
    count_block(ids, A, E, NB, align, capacity, ticket, blk_cnt, counts, offsets, err, blockIdx.x);
}

__global__ __launch_bounds__(256) void permute_scatter_kernel(const int32_t* __restrict__ ids, int A, int E,
                                                             int capacity, const int32_t* __restrict__ blk_base,
                                                             const int32_t* __restrict__ counts,
                                                             const int32_t* __restrict__ offsets,
                                                             int32_t* __restrict__ row_to_assign,
                                                             int32_t* __restrict__ assign_to_row,
                                                             int32_t* __restrict__ err) {
    scatter_block(ids, A, E, capacity, blk_base, counts, offsets, row_to_assign, assign_to_row, err, blockIdx.x,
                  gridDim.x);
}

// Several ops' count and scatter passes in one launch each: op o owns blocks
// [blk0[o], blk0[o + 1]) and its own workspace (ticket and chunk table).
struct PermOp {
    const int32_t* ids;
    int32_t *counts, *offsets, *row_to_assign, *assign_to_row, *err, *blk;
    unsigned* ticket;
    int32_t A, E, NB, align, capacity, pad;
};
struct PermBatch {
    PermOp op[MOE_MAX_OPS];
    int32_t blk0[MOE_MAX_OPS + 1];
    int32_t n;
};

__device__ __forceinline__ int batch_op(const PermBatch& b) {
    int o = 0;
    while (o + 1 < b.n && (int)blockIdx.x >= b.blk0[o + 1]) ++o;      // uniform
    return o;
}

__global__ __launch_bounds__(256) void permute_count_batch_kernel(const PermBatch b) {
    const int o = batch_op(b);
    const PermOp& p = b.op[o];
    count_block(p.ids, p.A, p.E, p.NB, p.align, p.capacity, p.ticket, p.blk, p.counts, p.offsets, p.err,
                (int)blockIdx.x - b.blk0[o]);
}

__global__ __launch_bounds__(256) void permute_scatter_batch_kernel(const PermBatch b) {
    const int o = batch_op(b);
    const PermOp& p = b.op[o];
    scatter_block(p.ids, p.A, p.E, p.capacity, p.blk, p.counts, p.offsets, p.row_to_assign, p.assign_to_row, p.err,
                  (int)blockIdx.x - b.blk0[o], p.NB);
}

// One wave per row, grid-stride over rows [0, offsets[E]).
__global__ __launch_bounds__(256) void permute_gather_kernel(const int32_t* __restrict__ counts,
                                                            const int32_t* __restrict__ offsets, int E, int k,
                                                            int capacity, const uint4* __restrict__ x,
                                                            int row_vecs, const float* __restrict__ xs,
                                                            int n_scales, int32_t* __restrict__ row_to_assign,
                                                            uint4* __restrict__ x_perm,
                                                            float* __restrict__ xs_perm) {
    extern __shared__ int32_t soff[];                         // [E+1] offsets, [E] counts
    for (int i = threadIdx.x; i <= E; i += 256) soff[i] = offsets[i];
    for (int i = threadIdx.x; i < E; i += 256) soff[E + 1 + i] = counts[i];
    __syncthreads();
    const int total = soff[E] < capacity ? soff[E] : capacity;
    const int lane = threadIdx.x & 63;
    const int waves = gridDim.x * 4;
    for (int r = blockIdx.x * 4 + (threadIdx.x >> 6); r < total; r += waves) {
        int lo = 0, hi = E - 1;                               // expert e with offsets[e] <= r < offsets[e+1]
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (soff[mid] <= r) lo = mid; else hi = mid - 1;
        }
        const bool valid = (r - soff[lo]) < soff[E + 1 + lo];
        const int a = valid ? row_to_assign[r] : -1;
        uint4* dst = x_perm + (size_t)r * row_vecs;
        if (a >= 0) {
            const uint4* src = x + (size_t)(a / k) * row_vecs;
            for (int v = lane; v < row_vecs; v += 64) dst[v] = src[v];
            if (xs_perm)
                for (int v = lane; v < n_scales; v += 64) xs_perm[(size_t)r * n_scales + v] = xs[(size_t)(a / k) * n_scales + v];
        } else {
            const uint4 z = make_uint4(0, 0, 0, 0);
            for (int v = lane; v < row_vecs; v += 64) dst[v] = z;
            if (xs_perm)
                for (int v = lane; v < n_scales; v += 64) xs_perm[(size_t)r * n_scales + v] = 0.f;
        }
    }
}

// Workspace: a 256-byte header (word 0: the count kernel's ticket counter),
// then the [chunks][E] counts / bases.
constexpr size_t kWsHeader = 256;

int num_chunks(int32_t T, int32_t top_k) {
    const int64_t A = (int64_t)T * top_k;
    return (int)((A + kChunk - 1) / kChunk);
}

}  // namespace

extern "C" size_t moe_permute_workspace_bytes(int32_t T, int32_t top_k, int32_t E_local) {
    if (T < 0 || top_k < 1 || E_local < 1) return 0;
    const int nb = num_chunks(T, top_k);
    return kWsHeader + (size_t)(nb > 0 ? nb : 1) * (size_t)E_local * sizeof(int32_t);
}

namespace {
moe_status_t check_permute(const int32_t* topk_ids, int32_t T, int32_t top_k, int32_t E_local, const void* x,
                           moe_dtype_t x_dtype, const float* x_scales, int32_t H, int32_t row_align,
                           int32_t capacity, const int32_t* counts, const int32_t* offsets,
                           const int32_t* row_to_assign, const int32_t* assign_to_row, const void* x_perm,
                           const float* x_perm_scales, const void* workspace, const int32_t* error_flag) {
    using moeapk_host::fail;
    if (T < 0 || top_k < 1 || top_k > 32) return fail(MOE_ERR_INVALID_ARG, "moe_permute: T=%d top_k=%d", T, top_k);
    if (E_local < 1 || E_local > 1024) return fail(MOE_ERR_UNSUPPORTED, "moe_permute: E_local=%d outside [1,1024]", E_local);
    if (row_align < 1 || row_align > 1024) return fail(MOE_ERR_INVALID_ARG, "moe_permute: row_align=%d", row_align);
    if (H < 128 || H % 128 != 0) return fail(MOE_ERR_UNSUPPORTED, "moe_permute: H=%d is not a positive multiple of 128", H);
    if (x_dtype != MOE_BF16 && x_dtype != MOE_FP8_E4M3)
        return fail(MOE_ERR_UNSUPPORTED, "moe_permute: x_dtype %d not supported", x_dtype);
    const bool fp8 = x_dtype == MOE_FP8_E4M3;
    const int64_t need = (int64_t)T * (top_k < E_local ? top_k : E_local) + (int64_t)E_local * (row_align - 1);
    if (capacity < need)
        return fail(MOE_ERR_CAPACITY, "moe_permute: capacity %d < T*min(k,E_local) + E_local*(row_align-1) = %lld",
                    capacity, (long long)need);
    if ((int64_t)T * top_k > (int64_t)INT32_MAX / 2) return fail(MOE_ERR_UNSUPPORTED, "moe_permute: T*top_k too large");
    if (!counts || !offsets || !row_to_assign || !assign_to_row || !workspace || !error_flag ||
        (T > 0 && !topk_ids) || (x_perm && !x))
        return fail(MOE_ERR_INVALID_ARG, "moe_permute: null pointer");
    if (fp8 && x_perm && (!x_scales || !x_perm_scales))
        return fail(MOE_ERR_INVALID_ARG, "moe_permute: fp8 activations need x_scales and x_perm_scales");
    return MOE_OK;
}

// The activation copy of one op (only when x_perm is requested).
moe_status_t launch_gather(const int32_t* counts, const int32_t* offsets, int32_t E_local, int32_t top_k,
                           int32_t capacity, const void* x, bool fp8, const float* x_scales, int32_t H,
                           int32_t* row_to_assign, void* x_perm, float* x_perm_scales, hipStream_t s) {
    const int row_bytes = fp8 ? H : 2 * H;
    int grid = (capacity + 3) / 4;
    if (grid > 4096) grid = 4096;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(permute_gather_kernel, dim3(grid), dim3(256), (2 * E_local + 1) * sizeof(int32_t), s, counts,
                       offsets, E_local, top_k, capacity, (const uint4*)x, row_bytes / 16, x_scales,
                       fp8 ? H / 128 : 0, row_to_assign, (uint4*)x_perm, fp8 ? x_perm_scales : nullptr);
    return MOE_OK;
}
}  // namespace

extern "C" moe_status_t moe_permute(const int32_t* topk_ids, int32_t T, int32_t top_k, int32_t E_local,
                                    const void* x, moe_dtype_t x_dtype, const float* x_scales, int32_t H,
                                    int32_t row_align, int32_t capacity, int32_t* counts, int32_t* offsets,
                                    int32_t* row_to_assign, int32_t* assign_to_row, void* x_perm,
                                    float* x_perm_scales, void* workspace, int32_t* error_flag, void* stream) {
    using moeapk_host::fail;
    moe_status_t st = check_permute(topk_ids, T, top_k, E_local, x, x_dtype, x_scales, H, row_align, capacity,
                                    counts, offsets, row_to_assign, assign_to_row, x_perm, x_perm_scales,
                                    workspace, error_flag);
    if (st != MOE_OK) return st;
    st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    const bool fp8 = x_dtype == MOE_FP8_E4M3;

    hipStream_t s = (hipStream_t)stream;
    const int A = T * top_k;
    const int nb = num_chunks(T, top_k);
    const int nb1 = nb > 0 ? nb : 1;                           // T == 0: one block writes zero counts
    unsigned* ticket = (unsigned*)workspace;
    int32_t* blk = (int32_t*)((char*)workspace + kWsHeader);
    hipLaunchKernelGGL(permute_count_kernel, dim3(nb1), dim3(kThreads), 2 * E_local * sizeof(int32_t), s, topk_ids,
                       A, E_local, nb1, row_align, capacity, ticket, blk, counts, offsets, error_flag);
    hipLaunchKernelGGL(permute_scatter_kernel, dim3(nb1), dim3(kThreads), 5 * E_local * sizeof(int32_t), s, topk_ids,
                       A, E_local, capacity, blk, counts, offsets, row_to_assign, assign_to_row, error_flag);
    if (!x_perm) {
        const hipError_t err = hipGetLastError();
        if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_permute: launch failed: %s", hipGetErrorString(err));
        return MOE_OK;
    }
    launch_gather(counts, offsets, E_local, top_k, capacity, x, fp8, x_scales, H, row_to_assign, x_perm, x_perm_scales,
                  s);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_permute: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}

extern "C" moe_status_t moe_permute_batch(const moe_permute_args* ops, int32_t n_ops, void* stream) {
    using moeapk_host::fail;
    if (!ops || n_ops < 1 || n_ops > MOE_MAX_OPS)
        return fail(MOE_ERR_INVALID_ARG, "moe_permute_batch: n_ops=%d outside [1,%d]", n_ops, MOE_MAX_OPS);
    PermBatch b;
    memset(&b, 0, sizeof(b));
    int64_t blocks = 0;
    int e_max = 1;
    for (int o = 0; o < n_ops; ++o) {
        const moe_permute_args& a = ops[o];
        const moe_status_t st = check_permute(a.topk_ids, a.T, a.top_k, a.E_local, a.x, a.x_dtype, a.x_scales, a.H,
                                              a.row_align, a.capacity, a.counts, a.offsets, a.row_to_assign,
                                              a.assign_to_row, a.x_perm, a.x_perm_scales, a.workspace,
                                              a.error_flag);
        if (st != MOE_OK) return st;
        const int nb = num_chunks(a.T, a.top_k);
        PermOp& p = b.op[o];
        p.ids = a.topk_ids;
        p.counts = a.counts;
        p.offsets = a.offsets;
        p.row_to_assign = a.row_to_assign;
        p.assign_to_row = a.assign_to_row;
        p.err = a.error_flag;
        p.ticket = (unsigned*)a.workspace;
        p.blk = (int32_t*)((char*)a.workspace + kWsHeader);
        p.A = a.T * a.top_k;
        p.E = a.E_local;
        p.NB = nb > 0 ? nb : 1;                                 // T == 0: one block writes zero counts
        p.align = a.row_align;
        p.capacity = a.capacity;
        b.blk0[o] = (int32_t)blocks;
        blocks += p.NB;
        e_max = a.E_local > e_max ? a.E_local : e_max;
    }
    if (blocks > INT32_MAX) return fail(MOE_ERR_UNSUPPORTED, "moe_permute_batch: too many assignments");
    b.blk0[n_ops] = (int32_t)blocks;
    b.n = n_ops;
    moe_status_t st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    hipLaunchKernelGGL(permute_count_batch_kernel, dim3((unsigned)blocks), dim3(kThreads),
                       2 * e_max * sizeof(int32_t), s, b);
    hipLaunchKernelGGL(permute_scatter_batch_kernel, dim3((unsigned)blocks), dim3(kThreads),
                       5 * e_max * sizeof(int32_t), s, b);
    for (int o = 0; o < n_ops; ++o) {
        const moe_permute_args& a = ops[o];
        if (a.x_perm)
            launch_gather(a.counts, a.offsets, a.E_local, a.top_k, a.capacity, a.x, a.x_dtype == MOE_FP8_E4M3,
                          a.x_scales, a.H, a.row_to_assign, a.x_perm, a.x_perm_scales, s);
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_permute_batch: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}
