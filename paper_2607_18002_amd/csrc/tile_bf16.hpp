// bf16 grouped-GEMM tile on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// One 256-thread workgroup computes a BM x BN output tile over the full K.
// The four waves split the BN columns (BN/4 each) and all share the BM rows:
//  * B (weight rows, K-contiguous) is private to a wave, so it streams from
//    global memory straight into MFMA operand registers, double-buffered
//    (two K steps in flight per wave), with no LDS round trip;
//  * A (activation rows, shared by the four waves) is staged through LDS,
//    double-buffered, with rows padded by 16 bytes so an operand read is free
//    of bank conflicts.
// K order: K runs in 64-element chunks; in each chunk lanes 0-31 take
// elements [0, 32) and lanes 32-63 take [32, 64), 8 per MFMA, so MFMA kk of a
// K step covers chunk kk/4, elements (lane/32)*32 + (kk%4)*8 .. +8.  A and B
// use the same order; the sum over K is unchanged.
//
// GLU tiles (GEMM-1) take BN/2 gate rows and BN/2 up rows of the [2I, H]
// gate/up matrix; every wave holds a gate block and the up block of the same
// columns, so h = silu(g) * u is formed lane-locally in the epilogue.
// MACT, the number of 32-row blocks with valid rows, is a template argument:
// the K loop is branch-free and blocks past the valid rows cost nothing.
#pragma once

#include "common.hpp"

namespace moeapk {

template <int BM_, int BN_, int BK_>
struct TileShape {
    static constexpr int BM = BM_, BN = BN_, BK = BK_;
    static constexpr int MB = BM / 32;               // 32-row blocks
    static constexpr int WCOLS = BN / 4;             // B rows (output columns) per wave
    static constexpr int NBW = WCOLS / 32;           // 32-column MFMA blocks per wave
    static constexpr int KK = BK / 16;               // MFMAs along K per K step
    static constexpr int LDS_ROW = BK * 2 + 16;      // bytes per LDS row of A
    static constexpr int A_STAGE = BM * LDS_ROW;
    static constexpr int LDS = 2 * A_STAGE;
    static constexpr int CPR = BK / 8;               // 16-byte chunks per A row and K step
    static constexpr int RPP = 256 / CPR;            // A rows loaded per pass of 256 threads
    static_assert(NBW >= 2 && NBW % 2 == 0, "GLU needs a gate and an up block per wave");
    static_assert(256 % CPR == 0 && RPP <= 32 && 32 % RPP == 0, "an A load pass stays inside one 32-row block");
};

template <class S, int MACT>
struct TileRegs {
    static constexpr int CA = MACT * 32 / S::RPP;    // A chunks per thread and K step
};

// Raw buffer loads: the tile's base address lives in an SGPR descriptor, the
// per-lane offset in one VGPR, the K-step offset in an SGPR and the per-MFMA
// offset in the instruction, so a load needs no address arithmetic.  The
// descriptor's size bounds the tile's extent (reads past it return zero).
constexpr int kBufferWord3 = 0x00020000;   // gfx9-family raw buffer: 32-bit data format, no swizzle

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferWord3);
}

template <int CA>
__device__ __forceinline__ void load_a(u32x4 (&ra)[CA], __amdgpu_buffer_rsrc_t A, const uint32_t (&aoff)[CA],
                                       int k0b) {
#pragma unroll
    for (int i = 0; i < CA; ++i) ra[i] = __builtin_amdgcn_raw_buffer_load_b128(A, (int)aoff[i], k0b, 0);
}

template <int CA>
__device__ __forceinline__ void store_a(char* buf, const u32x4 (&ra)[CA], const uint32_t (&alds)[CA]) {
#pragma unroll
    for (int i = 0; i < CA; ++i) *(u32x4*)(buf + alds[i]) = ra[i];
}

// Weight fragments of one K step.  Row-major weights: lane reads 16 bytes of
// its row per MFMA (k0b = step * BK * 2).  Packed weights (moe_pack_weights):
// each 32-row x 64-element chunk is 4 KB laid out as [kk%4][lane][16 B], so
// each load instruction reads 1 KB contiguous (k0b = step * BK * 64).
template <class S, bool PACKED>
__device__ __forceinline__ void load_b(bf16x8 (&rb)[S::NBW][S::KK], __amdgpu_buffer_rsrc_t B,
                                       const uint32_t (&boff)[S::NBW], int k0b) {
#pragma unroll
    for (int j = 0; j < S::NBW; ++j)
#pragma unroll
        for (int kk = 0; kk < S::KK; ++kk) {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(
                B, (int)(boff[j] + (PACKED ? kk * 1024 : (kk >> 2) * 128 + (kk & 3) * 16)), k0b, 0);
            rb[j][kk] = __builtin_bit_cast(bf16x8, v);
        }
}

// One K step of MFMAs.  The A fragments of step kk+1 are read from LDS while
// the MFMAs of step kk run (two register sets), and the scheduling-group
// barriers keep that order: each step is {MACT LDS reads, MACT*NBW MFMAs}.
template <class S, int MACT>
__device__ __forceinline__ void mma_step(f32x16 (&acc)[MACT][S::NBW], const bf16x8 (&rb)[S::NBW][S::KK],
                                         const char* buf, int lane) {
    const char* arow = buf + (lane & 31) * S::LDS_ROW + (lane >> 5) * 64;   // lanes 32-63: +32 elements
    bf16x8 af[2][MACT];
#pragma unroll
    for (int i = 0; i < MACT; ++i) af[0][i] = *(const bf16x8*)(arow + i * 32 * S::LDS_ROW);
    __builtin_amdgcn_sched_group_barrier(0x100, MACT, 0);                              // DS reads of step 0
#pragma unroll
    for (int kk = 0; kk < S::KK; ++kk) {
        const int cur = kk & 1;
        if (kk + 1 < S::KK) {
#pragma unroll
            for (int i = 0; i < MACT; ++i)
                af[cur ^ 1][i] = *(const bf16x8*)(arow + i * 32 * S::LDS_ROW + ((kk + 1) >> 2) * 128 + ((kk + 1) & 3) * 16);
        }
#pragma unroll
        for (int i = 0; i < MACT; ++i)
#pragma unroll
            for (int j = 0; j < S::NBW; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], rb[j][kk], acc[i][j], 0, 0, 0);
        if (kk + 1 < S::KK) __builtin_amdgcn_sched_group_barrier(0x100, MACT, 0);   // DS reads of kk+1
        __builtin_amdgcn_sched_group_barrier(0x008, MACT * S::NBW, 0);                // MFMAs of kk
    }
}

// A   : tile row 0 at k = 0, row stride lda elements; rows [0, 32*MACT) are read
// B   : first B row of the tile (GLU: gate row n0), row stride ldb elements
// up_rows : GLU only, rows from the gate block to the matching up block (I)
// out : output tile origin, row stride ldo (bf16); rows [0, 32*MACT) written
template <class S, bool GLU, int MACT, bool PACKED = false>
__device__ __forceinline__ void gemm_tile_bf16(const uint16_t* __restrict__ A, int lda,
                                               const uint16_t* __restrict__ B, int ldb, int up_rows, int K,
                                               uint16_t* __restrict__ out, int ldo, char* lds) {
    constexpr int CA = TileRegs<S, MACT>::CA;
    const int tid = threadIdx.x, lane = tid & 63, wn = tid >> 6;

    uint32_t boff[S::NBW];
#pragma unroll
    for (int j = 0; j < S::NBW; ++j) {
        int row;
        if (GLU) {
            constexpr int half = S::NBW / 2;
            const int jj = j < half ? j : j - half;
            row = wn * (S::WCOLS / 2) + 32 * jj + (lane & 31) + (j < half ? 0 : up_rows);
        } else {
            row = wn * S::WCOLS + 32 * j + (lane & 31);
        }
        if (PACKED)   // row is 32-aligned minus the lane part; the block starts where row-major row (row & ~31) would
            boff[j] = (uint32_t)(row - (lane & 31)) * (uint32_t)ldb * 2u + (uint32_t)(lane * 16);
        else
            boff[j] = (uint32_t)row * (uint32_t)ldb * 2u + (uint32_t)((lane >> 5) * 64);
    }
    uint32_t aoff[CA], alds[CA];
#pragma unroll
    for (int i = 0; i < CA; ++i) {
        const int idx = tid + 256 * i, r = idx / S::CPR, c = idx % S::CPR;
        aoff[i] = (uint32_t)r * (uint32_t)lda * 2u + c * 16;
        alds[i] = r * S::LDS_ROW + c * 16;
    }
    // extents: A rows [0, 32*MACT); B rows [0, BN) or, for GLU, gate rows [0, BN/2) and up rows [up_rows, up_rows + BN/2)
    const __amdgpu_buffer_rsrc_t Ab = make_rsrc(A, (uint32_t)(MACT * 32) * (uint32_t)lda * 2u);
    const __amdgpu_buffer_rsrc_t Bb =
        make_rsrc(B, (uint32_t)(GLU ? up_rows + S::BN / 2 : S::BN) * (uint32_t)ldb * 2u);
    char* lds0 = lds;
    char* lds1 = lds + S::A_STAGE;

    f32x16 acc[MACT][S::NBW];
#pragma unroll
    for (int i = 0; i < MACT; ++i)
#pragma unroll
        for (int j = 0; j < S::NBW; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    u32x4 ra[CA];
    bf16x8 rb0[S::NBW][S::KK], rb1[S::NBW][S::KK];
    const int nk = K / S::BK;
    constexpr int KB = S::BK * 2;                     // bytes per K step of a row-major row
    constexpr int KBB = PACKED ? S::BK * 64 : KB;     // bytes per K step of a weight fragment stream
    static_assert(S::BK % 64 == 0, "K steps are whole 64-element chunks");

    // K is a multiple of 2*BK (checked by the host), so the loop runs whole pairs of K steps.
    // A loads are issued before the B loads of the same K step: staging A into
    // LDS then waits only for A (vmcnt counts in issue order) and leaves the
    // later B loads in flight.
    load_a<CA>(ra, Ab, aoff, 0);
    load_b<S, PACKED>(rb0, Bb, boff, 0);
    store_a<CA>(lds0, ra, alds);
    load_a<CA>(ra, Ab, aoff, KB);
    load_b<S, PACKED>(rb1, Bb, boff, KBB);
    __syncthreads();
    for (int s = 0; s < nk; s += 2) {
        const bool more = s + 2 < nk;
        mma_step<S, MACT>(acc, rb0, lds0, lane);
        store_a<CA>(lds1, ra, alds);
        if (more) {
            load_a<CA>(ra, Ab, aoff, (s + 2) * KB);
            load_b<S, PACKED>(rb0, Bb, boff, (s + 2) * KBB);
        }
        __syncthreads();
        mma_step<S, MACT>(acc, rb1, lds1, lane);
        if (more) {
            store_a<CA>(lds0, ra, alds);
            load_a<CA>(ra, Ab, aoff, (s + 3) * KB);
            load_b<S, PACKED>(rb1, Bb, boff, (s + 3) * KBB);
        }
        __syncthreads();
    }

    // Epilogue.  32x32 accumulator layout: lane holds column (lane & 31) and
    // rows (r/4)*8 + (lane/32)*4 + r%4 of its block, r = 0..15.
#pragma unroll
    for (int i = 0; i < MACT; ++i) {
        const int row_base = 32 * i + (lane >> 5) * 4;
        if (GLU) {
#pragma unroll
            for (int j = 0; j < S::NBW / 2; ++j) {
                const int col = wn * (S::WCOLS / 2) + 32 * j + (lane & 31);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float g = acc[i][j][r], u = acc[i][j + S::NBW / 2][r];
                    const float hv = g / (1.f + __expf(-g)) * u;
                    out[(long)(row_base + (r >> 2) * 8 + (r & 3)) * ldo + col] = (uint16_t)f2bf_bits(hv);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < S::NBW; ++j) {
                const int col = wn * S::WCOLS + 32 * j + (lane & 31);
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    out[(long)(row_base + (r >> 2) * 8 + (r & 3)) * ldo + col] = (uint16_t)f2bf_bits(acc[i][j][r]);
            }
        }
    }
}

// Dispatch on the number of 32-row blocks holding valid rows (uniform per tile).
template <class S, bool GLU, bool PACKED>
__device__ __forceinline__ void gemm_tile_bf16_rows(int rows32, const uint16_t* A, int lda, const uint16_t* B, int ldb,
                                                    int up_rows, int K, uint16_t* out, int ldo, char* lds) {
    static_assert(S::MB == 4, "dispatch written for 128-row tiles");
    switch (rows32 >> 5) {
        case 1: gemm_tile_bf16<S, GLU, 1, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds); break;
        case 2: gemm_tile_bf16<S, GLU, 2, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds); break;
        case 3: gemm_tile_bf16<S, GLU, 3, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds); break;
        default: gemm_tile_bf16<S, GLU, 4, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds); break;
    }
}

}  // namespace moeapk
