// a7: weighted combine back to token order (Background, "MoE LLM Inference":
// the chosen experts' outputs are combined before the next layer).
//
// One 128-thread block per token; each thread owns 8 consecutive columns
// (one 16-byte bf16 vector) per pass and accumulates the token's local slots in
// ascending slot order in fp32.  Slot rows and weights are block-uniform.
#include <cstring>

#include "common.hpp"

namespace {

template <bool OUT_BF16>
__device__ __forceinline__ void combine_token(const uint4* __restrict__ y_perm,
                                              const int32_t* __restrict__ assign_to_row,
                                              const float* __restrict__ topk_w, int k, int vecs,
                                              void* __restrict__ y, int t) {
    const int32_t* rows = assign_to_row + (size_t)t * k;
    const float* w = topk_w + (size_t)t * k;
    for (int v = threadIdx.x; v < vecs; v += blockDim.x) {
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (int j = 0; j < k; ++j) {
            const int r = rows[j];
            if (r < 0) continue;
            const float wj = w[j];
            const uint4 q = y_perm[(size_t)r * vecs + v];
            const uint32_t p[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc[2 * i] = fmaf(wj, moeapk::bf_bits2f(p[i] & 0xFFFFu), acc[2 * i]);
                acc[2 * i + 1] = fmaf(wj, moeapk::bf_bits2f(p[i] >> 16), acc[2 * i + 1]);
            }
        }
        if (OUT_BF16) {
            uint4 o;
            o.x = moeapk::f2bf_bits(acc[0]) | (moeapk::f2bf_bits(acc[1]) << 16);
            o.y = moeapk::f2bf_bits(acc[2]) | (moeapk::f2bf_bits(acc[3]) << 16);
            o.z = moeapk::f2bf_bits(acc[4]) | (moeapk::f2bf_bits(acc[5]) << 16);
            o.w = moeapk::f2bf_bits(acc[6]) | (moeapk::f2bf_bits(acc[7]) << 16);
            ((uint4*)y)[(size_t)t * vecs + v] = o;
        } else {
            float4* out = (float4*)y + ((size_t)t * vecs + v) * 2;
            out[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
            out[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
        }
    }
}

template <bool OUT_BF16>
__global__ __launch_bounds__(128) void combine_kernel(const uint4* __restrict__ y_perm,
                                                     const int32_t* __restrict__ assign_to_row,
                                                     const float* __restrict__ topk_w, int k, int vecs,
                                                     void* __restrict__ y) {
    combine_token<OUT_BF16>(y_perm, assign_to_row, topk_w, k, vecs, y, blockIdx.x);
}

// Several ops in one launch: op o owns blocks (tokens) [blk0[o], blk0[o + 1]).
struct CombineBatch {
    moe_combine_args op[MOE_MAX_OPS];
    int32_t blk0[MOE_MAX_OPS + 1];
    int32_t n;
};

template <bool OUT_BF16>
__global__ __launch_bounds__(128) void combine_batch_kernel(const CombineBatch b) {
    int o = 0;
    while (o + 1 < b.n && (int)blockIdx.x >= b.blk0[o + 1]) ++o;      // uniform
    const moe_combine_args& a = b.op[o];
    combine_token<OUT_BF16>((const uint4*)a.y_perm, a.assign_to_row, a.topk_w, a.top_k, a.H / 8, a.y,
                            (int)blockIdx.x - b.blk0[o]);
}

moe_status_t check_combine(const void* y_perm, const int32_t* assign_to_row, const float* topk_w, int32_t T,
                           int32_t top_k, int32_t H, const void* y, moe_dtype_t y_dtype) {
    using moeapk_host::fail;
    if (T < 0 || top_k < 1 || top_k > 32) return fail(MOE_ERR_INVALID_ARG, "moe_combine: T=%d top_k=%d", T, top_k);
    if (H < 8 || H % 8 != 0) return fail(MOE_ERR_UNSUPPORTED, "moe_combine: H=%d not a positive multiple of 8", H);
    if (y_dtype != MOE_BF16 && y_dtype != MOE_F32)
        return fail(MOE_ERR_UNSUPPORTED, "moe_combine: y_dtype %d not supported", y_dtype);
    if (T > 0 && (!y_perm || !assign_to_row || !topk_w || !y)) return fail(MOE_ERR_INVALID_ARG, "moe_combine: null pointer");
    return MOE_OK;
}

}  // namespace

extern "C" moe_status_t moe_combine(const void* y_perm, const int32_t* assign_to_row, const float* topk_w,
                                    int32_t T, int32_t top_k, int32_t H, void* y, moe_dtype_t y_dtype,
                                    void* stream) {
    using moeapk_host::fail;
    moe_status_t st = check_combine(y_perm, assign_to_row, topk_w, T, top_k, H, y, y_dtype);
    if (st != MOE_OK) return st;
    if (T == 0) return MOE_OK;
    st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    const int vecs = H / 8;
    if (y_dtype == MOE_BF16)
        hipLaunchKernelGGL(combine_kernel<true>, dim3(T), dim3(128), 0, s, (const uint4*)y_perm, assign_to_row, topk_w,
                           top_k, vecs, y);
    else
        hipLaunchKernelGGL(combine_kernel<false>, dim3(T), dim3(128), 0, s, (const uint4*)y_perm, assign_to_row,
                           topk_w, top_k, vecs, y);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_combine: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}

extern "C" moe_status_t moe_combine_batch(const moe_combine_args* ops, int32_t n_ops, void* stream) {
    using moeapk_host::fail;
    if (!ops || n_ops < 1 || n_ops > MOE_MAX_OPS)
        return fail(MOE_ERR_INVALID_ARG, "moe_combine_batch: n_ops=%d outside [1,%d]", n_ops, MOE_MAX_OPS);
    CombineBatch b;
    memset(&b, 0, sizeof(b));
    int64_t blocks = 0;
    for (int o = 0; o < n_ops; ++o) {
        const moe_combine_args& a = ops[o];
        const moe_status_t st = check_combine(a.y_perm, a.assign_to_row, a.topk_w, a.T, a.top_k, a.H, a.y, a.y_dtype);
        if (st != MOE_OK) return st;
        if (a.y_dtype != ops[0].y_dtype)
            return fail(MOE_ERR_INVALID_ARG, "moe_combine_batch: entries %d and 0 differ in y_dtype", o);
        b.op[o] = a;
        b.blk0[o] = (int32_t)blocks;
        blocks += a.T;
    }
    if (blocks > INT32_MAX) return fail(MOE_ERR_UNSUPPORTED, "moe_combine_batch: too many tokens");
    b.blk0[n_ops] = (int32_t)blocks;
    b.n = n_ops;
    if (blocks == 0) return MOE_OK;
    moe_status_t st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    if (ops[0].y_dtype == MOE_BF16)
        hipLaunchKernelGGL(combine_batch_kernel<true>, dim3((unsigned)blocks), dim3(128), 0, s, b);
    else
        hipLaunchKernelGGL(combine_batch_kernel<false>, dim3((unsigned)blocks), dim3(128), 0, s, b);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_combine_batch: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}
