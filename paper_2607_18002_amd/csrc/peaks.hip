// Measurement kernels for the achievable peaks of one MI355X (gfx950), against
// which the hot path's kernels are also reported (context, beside the vendor
// peaks):
//  - an MFMA loop: every wave issues independent v_mfma_f32_32x32x16_bf16
//    (or v_mfma_scale_f32_32x32x64_f8f6f4) back to back on register operands,
//    nothing else, so the time is the matrix pipes' throughput at whatever
//    clock the chip holds under that load;
//  - a streaming read of a known number of bytes with 16-byte loads (the width
//    the FFN tiles use), many loads in flight per lane, one word written per
//    workgroup: its bytes per second are the achievable HBM read rate, and its
//    FETCH_SIZE counter calibrates the counter against a known byte count.
// Built into libmoe_peaks.so, separate from the hot-path library.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;   // independent accumulators per wave

__global__ __launch_bounds__(256) void mfma_bf16_loop(int iters, float* out) {
    const int tid = threadIdx.x;
    bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(0.001f * (float)((tid + i) & 7));
        b[i] = (__bf16)(0.001f * (float)((tid * 3 + i) & 7));
    }
    f32x16 acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[c][r];
    out[blockIdx.x * 256 + tid] = s;
}

__global__ __launch_bounds__(256) void mfma_fp8_loop(int iters, float* out) {
    const int tid = threadIdx.x;
    i32x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = 0x38383838 ^ ((tid + i) & 3);    // small e4m3 values
        b[i] = 0x30303030 ^ ((tid * 5 + i) & 3);
    }
    f32x16 acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < kChains; ++c)
            acc[c] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc[c], 0, 0, 0, 127, 0, 127);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[c][r];
    out[blockIdx.x * 256 + tid] = s;
}

// Reads words [0, n16) of src (16 bytes each), grid-strided with kUnroll loads
// in flight per lane; writes one xor word per workgroup.
constexpr int kUnroll = 8;
__global__ __launch_bounds__(256) void stream_read(const u32x4* __restrict__ src, int64_t n16, uint32_t* sink) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    uint32_t x = 0;
    for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n16; i += stride) {
        const u32x4 v = src[i];
        x ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    __shared__ uint32_t red[256];
    red[threadIdx.x] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int j = 0; j < 256; ++j) t ^= red[j];
        sink[blockIdx.x] = t;
    }
}

}  // namespace

extern "C" {

// MFMA loop: `blocks` workgroups of 4 waves, `iters` rounds of 8 MFMAs per
// wave.  dtype 1 = bf16 (32x32x16: 32768 flop each), 2 = fp8 (32x32x64: 131072
// flop each).  out: blocks*256 floats.  Returns 0, or -1 on bad arguments /
// a launch error.
int32_t moe_peak_mfma(int32_t dtype, int32_t blocks, int32_t iters, float* out, void* stream) {
    if (blocks < 1 || iters < 1 || !out || (dtype != 1 && dtype != 2)) return -1;
    hipStream_t s = (hipStream_t)stream;
    if (dtype == 1) hipLaunchKernelGGL(mfma_bf16_loop, dim3(blocks), dim3(256), 0, s, iters, out);
    else hipLaunchKernelGGL(mfma_fp8_loop, dim3(blocks), dim3(256), 0, s, iters, out);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Streaming read of `bytes` (a multiple of 16) from src with `blocks`
// workgroups; sink: blocks uint32 words.
int32_t moe_peak_stream_read(const void* src, int64_t bytes, int32_t blocks, uint32_t* sink, void* stream) {
    if (!src || !sink || bytes < 16 || bytes % 16 != 0 || blocks < 1) return -1;
    hipLaunchKernelGGL(stream_read, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (const u32x4*)src, bytes / 16,
                       sink);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // extern "C"
