// One-time relayout of expert weights into the order the FFN kernel streams
// them (see moe_pack_weights in moe_apk.h).  Not on the hot path.
#include "common.hpp"

namespace {

// One thread per 16-byte unit of the packed matrix.
__global__ __launch_bounds__(256) void pack_bf16_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                       long units, int N, int K) {
    const long per_matrix = (long)N * K / 8;                 // 16-byte units per [N, K] matrix
    const int chunks = K / 64;
    for (long u = (long)blockIdx.x * 256 + threadIdx.x; u < units; u += (long)gridDim.x * 256) {
        const long e = u / per_matrix;
        long r = u - e * per_matrix;
        const int lane = (int)(r & 63);
        r >>= 6;
        const int q = (int)(r & 3);
        r >>= 2;
        const int c = (int)(r % chunks);
        const long b = r / chunks;
        const long row = b * 32 + (lane & 31);
        const long col = (long)c * 64 + (lane >> 5) * 32 + q * 8;
        dst[u] = src[e * per_matrix + (row * K + col) / 8];
    }
}

// fp8 codes: per 32-row block and 128-element K chunk, 4 KB laid out as
// [kk][half][lane][16 B]; lane `lane` holds row 32*b + lane%32, elements
// 128*c + 64*kk + (lane/32)*32 + 16*half .. +16.
__global__ __launch_bounds__(256) void pack_fp8_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                      long units, int N, int K) {
    const long per_matrix = (long)N * K / 16;                // 16-byte units per [N, K] matrix
    const int chunks = K / 128;
    for (long u = (long)blockIdx.x * 256 + threadIdx.x; u < units; u += (long)gridDim.x * 256) {
        const long e = u / per_matrix;
        long r = u - e * per_matrix;
        const int lane = (int)(r & 63);
        r >>= 6;
        const int half = (int)(r & 1);
        r >>= 1;
        const int kk = (int)(r & 1);
        r >>= 1;
        const int c = (int)(r % chunks);
        const long b = r / chunks;
        const long row = b * 32 + (lane & 31);
        const long col = (long)c * 128 + kk * 64 + (lane >> 5) * 32 + half * 16;
        dst[u] = src[e * per_matrix + (row * K + col) / 16];
    }
}

}  // namespace

extern "C" moe_status_t moe_pack_weights(const void* src, void* dst, int32_t E, int32_t N, int32_t K,
                                         moe_dtype_t dtype, void* stream) {
    using moeapk_host::fail;
    if (dtype != MOE_BF16 && dtype != MOE_FP8_E4M3)
        return fail(MOE_ERR_UNSUPPORTED, "moe_pack_weights: dtype %d not supported", dtype);
    const int kq = dtype == MOE_BF16 ? 64 : 128;             // K elements per packed chunk
    if (E < 1 || N < 32 || K < kq || N % 32 != 0 || K % kq != 0)
        return fail(MOE_ERR_UNSUPPORTED, "moe_pack_weights: E=%d N=%d K=%d (need N%%32 == 0, K%%%d == 0)", E, N, K, kq);
    if (!src || !dst) return fail(MOE_ERR_INVALID_ARG, "moe_pack_weights: null pointer");
    if (src == dst) return fail(MOE_ERR_INVALID_ARG, "moe_pack_weights: src and dst must not alias");
    moe_status_t st = moeapk_host::check_device();
    if (st != MOE_OK) return st;
    const long units = (long)E * N * K / (dtype == MOE_BF16 ? 8 : 16);
    long grid = (units + 255) / 256;
    if (grid > 65536) grid = 65536;
    if (dtype == MOE_BF16)
        hipLaunchKernelGGL(pack_bf16_kernel, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream, (const uint4*)src,
                           (uint4*)dst, units, N, K);
    else
        hipLaunchKernelGGL(pack_fp8_kernel, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream, (const uint4*)src,
                           (uint4*)dst, units, N, K);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(MOE_ERR_HIP, "moe_pack_weights: launch failed: %s", hipGetErrorString(err));
    return MOE_OK;
}
