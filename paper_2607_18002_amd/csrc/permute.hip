// a2: permutation into per-expert contiguous segments at final offsets
// (Background, "Prefill-Decode Disaggregation": contiguous layout;
// "One-Sided Dispatch and Combine": each expert's destination and final offset
// are fixed after routing, before the activations are written).
//
// Four launches on the caller's stream:
//   count   : per-chunk expert histogram in LDS (512 assignments per block)
//   scan    : expert counts, padded segment offsets, per-(chunk, expert) bases;
//             each expert's prefix over chunks is split across 1024/E threads
//   scatter : stable rank of every assignment inside its chunk, built from
//             wave ballots (rank = popcount(match & lanes-below)) plus per-wave
//             and per-iteration running counts -> row_to_assign / assign_to_row.
//             The result is the unique order "ascending assignment a = t*k+j",
//             so it is bit-exact and independent of scheduling.
//   gather  : one wave per row copies x[a / k] (16-byte vectors) into x_perm,
//             zero-fills padding rows and marks them -1; without x_perm (the
//             FFN then gathers its rows itself) it only marks padding rows.
#include "common.hpp"

namespace {

using moeapk::set_status;

constexpr int kThreads = 256;
constexpr int kIters = 2;
constexpr int kChunk = kThreads * kIters;   // assignments per block

__global__ __launch_bounds__(256) void permute_count_kernel(const int32_t* __restrict__ ids, int A, int E,
                                                           int32_t* __restrict__ blk_cnt,
                                                           int32_t* __restrict__ err) {
    extern __shared__ int32_t hist[];
    for (int e = threadIdx.x; e < E; e += kThreads) hist[e] = 0;
    __syncthreads();
    const int base = blockIdx.x * kChunk;
    for (int it = 0; it < kIters; ++it) {
        const int a = base + it * kThreads + threadIdx.x;
        if (a < A) {
            const int id = ids[a];
            if (id < -1 || id >= E) set_status(err, MOE_ERR_BAD_EXPERT);
            else if (id >= 0) atomicAdd(&hist[id], 1);
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += kThreads) blk_cnt[(size_t)blockIdx.x * E + e] = hist[e];
}

__global__ __launch_bounds__(1024) void permute_scan_kernel(int NB, int E, int align, int capacity,
                                                           int32_t* __restrict__ blk_cnt,   // in: counts; out: bases
                                                           int32_t* __restrict__ counts,
                                                           int32_t* __restrict__ offsets,
                                                           int32_t* __restrict__ err) {
    __shared__ int32_t part[1024];       // per thread: the sum of its run of chunks, then its run's base
    __shared__ int32_t padded[1024];
    __shared__ int32_t scan[1024];
    // P threads per expert (P = 1024 / E rounded down to a power of two); thread
    // (e, j) owns chunks [j*R, (j+1)*R) of expert e, R = ceil(NB / P).
    int P = 1;
    while (P * 2 * E <= 1024) P *= 2;
    const int R = (NB + P - 1) / P;
    const int t = threadIdx.x, e = t / P, j = t - e * P;
    const bool mine = e < E;
    const int b0 = mine ? j * R : 0, b1 = mine ? min(NB, b0 + R) : 0;
    int sum = 0;
    for (int b = b0; b < b1; ++b) sum += blk_cnt[(size_t)b * E + e];
    part[t] = sum;
    __syncthreads();
    if (mine && j == 0) {                                      // exclusive prefix over the expert's P runs
        int run = 0;
        for (int q = 0; q < P; ++q) { const int v = part[t + q]; part[t + q] = run; run += v; }
        scan[e] = run;                                         // total rows of expert e (temporarily)
    }
    __syncthreads();
    const int tot = (t < E) ? scan[t] : 0;
    if (t < E) counts[t] = tot;
    padded[t] = (t < E) ? ((tot + align - 1) / align) * align : 0;
    __syncthreads();
    scan[t] = padded[t];
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {                 // inclusive Hillis-Steele scan over experts
        const int v = (t >= off) ? scan[t - off] : 0;
        __syncthreads();
        scan[t] += v;
        __syncthreads();
    }
    if (t < E) offsets[t] = scan[t] - padded[t];
    if (t == E - 1) {
        offsets[E] = scan[t];
        if (scan[t] > capacity) set_status(err, MOE_ERR_CAPACITY);
    }
    if (mine) {                                                // bases of this thread's chunks
        int run = scan[e] - padded[e] + part[t];
        for (int b = b0; b < b1; ++b) {
            const int c = blk_cnt[(size_t)b * E + e];
            blk_cnt[(size_t)b * E + e] = run;
            run += c;
        }
    }
}

__global__ __launch_bounds__(256) void permute_scatter_kernel(const int32_t* __restrict__ ids, int A, int E,
                                                             int capacity, const int32_t* __restrict__ blk_base,
                                                             int32_t* __restrict__ row_to_assign,
                                                             int32_t* __restrict__ assign_to_row,
                                                             int32_t* __restrict__ err) {
    extern __shared__ int32_t sm[];
    int32_t* running = sm;           // [E]   rows handed out in earlier iterations
    int32_t* wcnt = sm + E;          // [4][E] per-wave counts of the current iteration
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int i = tid; i < 5 * E; i += kThreads) sm[i] = 0;
    __syncthreads();
    const int base = blockIdx.x * kChunk;
    const int32_t* my_base = blk_base + (size_t)blockIdx.x * E;
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
        if (!x_perm) {                                        // maps only
            if (a < 0 && lane == 0) row_to_assign[r] = -1;
            continue;
        }
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
            if (lane == 0) row_to_assign[r] = -1;
        }
    }
}

int num_chunks(int32_t T, int32_t top_k) {
    const int64_t A = (int64_t)T * top_k;
    return (int)((A + kChunk - 1) / kChunk);
}

}  // namespace

extern "C" size_t moe_permute_workspace_bytes(int32_t T, int32_t top_k, int32_t E_local) {
    if (T < 0 || top_k < 1 || E_local < 1) return 0;
    const int nb = num_chunks(T, top_k);
    return (size_t)(nb > 0 ? nb : 1) * (size_t)E_local * sizeof(int32_t) + 256;
}

extern "C" moe_status_t moe_permute(const int32_t* topk_ids, int32_t T, int32_t top_k, int32_t E_local,
                                    const void* x, moe_dtype_t x_dtype, const float* x_scales, int32_t H,
                                    int32_t row_align, int32_t capacity, int32_t* counts, int32_t* offsets,
                                    int32_t* row_to_assign, int32_t* assign_to_row, void* x_perm,
                                    float* x_perm_scales, void* workspace, int32_t* error_flag, void* stream) {
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
    moe_status_t st = moeapk_host::check_device();
    if (st != MOE_OK) return st;

    hipStream_t s = (hipStream_t)stream;
    const int A = T * top_k;
    const int nb = num_chunks(T, top_k);
    int32_t* blk = (int32_t*)workspace;
    if (nb > 0) {
        hipLaunchKernelGGL(permute_count_kernel, dim3(nb), dim3(kThreads), E_local * sizeof(int32_t), s, topk_ids, A,
                           E_local, blk, error_flag);
    }
    hipLaunchKernelGGL(permute_scan_kernel, dim3(1), dim3(1024), 0, s, nb, E_local, row_align, capacity, blk, counts,
                       offsets, error_flag);
    if (nb > 0) {
        hipLaunchKernelGGL(permute_scatter_kernel, dim3(nb), dim3(kThreads), 5 * E_local * sizeof(int32_t), s, topk_ids,
                           A, E_local, capacity, blk, row_to_assign, assign_to_row, error_flag);
    }
    const int row_bytes = fp8 ? H : 2 * H;
    const int rows_max = capacity;
    int grid = (rows_max + 3) / 4;
    if (grid > 4096) grid = 4096;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(permute_gather_kernel, dim3(grid), dim3(256), (2 * E_local + 1) * sizeof(int32_t), s, counts,
                       offsets, E_local, top_k, capacity, (const uint4*)x, row_bytes / 16, x_scales,
                       fp8 ? H / 128 : 0, row_to_assign, (uint4*)x_perm, (fp8 && x_perm) ? x_perm_scales : nullptr);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_permute: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}
