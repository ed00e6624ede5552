// Shared device helpers and host plumbing of the MoE hot-path library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moe_apk.h"

namespace moeapk {

// ----------------------------------------------------------------------------- vector types
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
// 16 bytes that may alias any other type: the epilogues stage results in LDS
// with 2- or 4-byte stores and read them back 16 bytes at a time, so the
// read-back must not be reordered above those stores by type-based aliasing.
typedef unsigned int u32x4_alias __attribute__((ext_vector_type(4), may_alias));

constexpr int kWave = 64;

// ----------------------------------------------------------------------------- conversions
// float -> bf16 bits, round to nearest even (gfx950's v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t f2bf_bits(float f) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
}
__device__ __forceinline__ float bf_bits2f(uint32_t h) { return __uint_as_float(h << 16); }

// ----------------------------------------------------------------------------- device status
// First error wins; never overwrites an earlier error.
__device__ __forceinline__ void set_status(int32_t* status, int32_t code) {
    if (status) atomicCAS(status, 0, code);
}

__device__ __forceinline__ uint64_t wall_ticks() { return wall_clock64(); }

// Wait until every global store this wave issued has reached the L2 (vmcnt = 0;
// expcnt and lgkmcnt left at their maxima).  A workgroup barrier alone does not
// do this, so waves that hand stores to another wave's release call it first.
__device__ __forceinline__ void wait_own_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Hardware register XCC_ID: the XCD a wave runs on.
__device__ __forceinline__ int xcc_id() {
    return __builtin_amdgcn_s_getreg((20) | (0 << 6) | (31 << 11)) & 0xF;
}

template <typename T>
__device__ __forceinline__ T ld_acquire_agent(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T ld_relaxed_agent(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T ld_acquire_system(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
}
template <typename T>
__device__ __forceinline__ void st_release_agent(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void st_release_system(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}
template <typename T>
__device__ __forceinline__ T add_release_agent(T* p, T v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T add_relaxed_agent(T* p, T v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ----------------------------------------------------------------------------- Eq. (3) / Eq. (4)
// Shared by host helpers and kernels so both compute the same integers.
__host__ __device__ __forceinline__ int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }

// Eq. (4) ("Online SM Reallocation") in workgroup units:
// q' = min(Q_max, ceil_c(q * x_moe / x*_moe)), ceil_c(n/d) = c * ceil(n / (d*c));
// x*_moe <= 0 selects the fixed quota (ratio 1).
__host__ __device__ __forceinline__ int32_t decode_quota(int32_t q, int32_t x_moe, int32_t x_star,
                                                         int32_t q_max, int32_t c) {
    int64_t num, den;
    if (x_star <= 0) { num = q; den = 1; }
    else { num = (int64_t)q * x_moe; den = x_star; }
    if (c < 1) c = 1;
    int64_t dc = den * c;
    int64_t r = (num <= 0) ? 0 : c * ((num + dc - 1) / dc);
    return (int32_t)(r < q_max ? r : q_max);
}

}  // namespace moeapk

// ----------------------------------------------------------------------------- host plumbing
namespace moeapk_host {
// Records a message for moe_last_error() and returns `code`.
moe_status_t fail(moe_status_t code, const char* fmt, ...);
// MOE_OK when the current device is gfx950; caches CU count and wall-clock rate.
moe_status_t check_device(int* cu_count = nullptr, int* wallclock_khz = nullptr);
}  // namespace moeapk_host
