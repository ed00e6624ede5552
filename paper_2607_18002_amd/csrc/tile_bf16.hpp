// bf16 grouped-GEMM tile on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// One 256-thread workgroup (4 waves in a WM x WN grid) computes a BM x BN
// output tile over the full K in BK steps.  Both operands are K-contiguous
// (A = activation rows, B = weight rows), so every global load is a 16-byte
// vector of one row and every MFMA operand is one 16-byte LDS read.
//
// Pipeline: global -> registers for step s+1 is issued before the MFMAs of
// step s; the registers are written to the other LDS buffer afterwards; one
// barrier per K step.  LDS rows are padded by 16 bytes so the 32 rows an MFMA
// operand spans fall on distinct banks.
//
// GLU tiles (GEMM-1) load BN/2 gate rows followed by BN/2 up rows of the
// [2I, H] gate/up matrix; each wave's gate and up accumulators cover the same
// output columns, so the SiLU(g)*u epilogue is lane-local.  Row blocks of 32
// that lie beyond the tile's valid rows are neither loaded nor computed.
#pragma once

#include "common.hpp"

namespace moeapk {

template <int BM_, int BN_, int BK_, int WM_, int WN_>
struct TileShape {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
    static constexpr int WTM = BM / WM;              // rows per wave
    static constexpr int MB = WTM / 32;              // 32-row MFMA blocks per wave
    static constexpr int NBW = BN / WN / 32;         // 32-column MFMA blocks per wave
    static constexpr int LDS_ROW = BK * 2 + 16;      // bytes per LDS row
    static constexpr int A_BYTES = BM * LDS_ROW;
    static constexpr int B_BYTES = BN * LDS_ROW;
    static constexpr int STAGE = A_BYTES + B_BYTES;
    static constexpr int LDS = 2 * STAGE;
    static constexpr int CPR = BK / 8;               // 16-byte chunks per row and K step
    static constexpr int CA = BM * CPR / 256;        // A chunks per thread and K step
    static constexpr int CB = BN * CPR / 256;        // B chunks per thread and K step
    static_assert(WM * WN == 4, "4 waves");
    static_assert(MB >= 1 && NBW >= 2 && NBW % 2 == 0, "tile shape");
    static_assert(CA * 256 == BM * CPR && CB * 256 == BN * CPR, "load split");
};

// B row (within the tile's BN rows) of the wave's j-th 32-column block.
template <class S, bool GLU>
__device__ __forceinline__ int b_block_row(int wn, int j) {
    if (GLU) {
        constexpr int half = S::BN / 2, per_wave = half / S::WN, nb2 = S::NBW / 2;
        return (j < nb2) ? wn * per_wave + 32 * j : half + wn * per_wave + 32 * (j - nb2);
    }
    return wn * (S::BN / S::WN) + 32 * j;
}

// A : tile row 0 at k = 0, row stride lda (elements)
// rows32 : rows to compute, a multiple of 32 in [32, BM]
// B : first B row of the tile (GLU: gate row n0), row stride ldb
// up_off : GLU only, element offset from the gate rows to the up rows
// out : output tile origin, row stride ldo (bf16)
template <class S, bool GLU>
__device__ __forceinline__ void gemm_tile_bf16(const uint16_t* __restrict__ A, int lda, int rows32,
                                               const uint16_t* __restrict__ B, int ldb, long up_off, int K,
                                               uint16_t* __restrict__ out, int ldo, char* lds) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / S::WN, wn = wave % S::WN;
    int mact = (rows32 - wm * S::WTM) / 32;
    mact = mact < 0 ? 0 : (mact > S::MB ? S::MB : mact);

    int a_goff[S::CA], a_loff[S::CA];
    bool a_ok[S::CA];
#pragma unroll
    for (int i = 0; i < S::CA; ++i) {
        const int idx = tid + 256 * i, r = idx / S::CPR, c = idx % S::CPR;
        a_ok[i] = r < rows32;
        a_goff[i] = r * lda + c * 8;
        a_loff[i] = r * S::LDS_ROW + c * 16;
    }
    long b_goff[S::CB];
    int b_loff[S::CB];
#pragma unroll
    for (int i = 0; i < S::CB; ++i) {
        const int idx = tid + 256 * i, r = idx / S::CPR, c = idx % S::CPR;
        long row_off;
        if (GLU) row_off = (r < S::BN / 2) ? (long)r * ldb : up_off + (long)(r - S::BN / 2) * ldb;
        else row_off = (long)r * ldb;
        b_goff[i] = row_off + c * 8;
        b_loff[i] = S::A_BYTES + r * S::LDS_ROW + c * 16;
    }

    uint4 ra[S::CA], rb[S::CB];
    f32x16 acc[S::MB][S::NBW];
#pragma unroll
    for (int i = 0; i < S::MB; ++i)
#pragma unroll
        for (int j = 0; j < S::NBW; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < S::CA; ++i)
            ra[i] = a_ok[i] ? *(const uint4*)(A + a_goff[i] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < S::CB; ++i) rb[i] = *(const uint4*)(B + b_goff[i] + k0);
    };
    auto sstore = [&](int buf) {
        char* base = lds + buf * S::STAGE;
#pragma unroll
        for (int i = 0; i < S::CA; ++i)
            if (a_ok[i]) *(uint4*)(base + a_loff[i]) = ra[i];
#pragma unroll
        for (int i = 0; i < S::CB; ++i) *(uint4*)(base + b_loff[i]) = rb[i];
    };
    auto compute = [&](int buf) {
        const char* base = lds + buf * S::STAGE;
#pragma unroll
        for (int kk = 0; kk < S::BK / 16; ++kk) {
            const int kofs = (kk * 16 + (lane >> 5) * 8) * 2;
            bf16x8 bfr[S::NBW];
#pragma unroll
            for (int j = 0; j < S::NBW; ++j)
                bfr[j] = *(const bf16x8*)(base + S::A_BYTES +
                                          (b_block_row<S, GLU>(wn, j) + (lane & 31)) * S::LDS_ROW + kofs);
#pragma unroll
            for (int i = 0; i < S::MB; ++i) {
                if (i < mact) {
                    const bf16x8 af =
                        *(const bf16x8*)(base + (wm * S::WTM + 32 * i + (lane & 31)) * S::LDS_ROW + kofs);
#pragma unroll
                    for (int j = 0; j < S::NBW; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bfr[j], acc[i][j], 0, 0, 0);
                }
            }
        }
    };

    const int nk = K / S::BK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int s = 0; s < nk; ++s) {
        if (s + 1 < nk) gload((s + 1) * S::BK);
        compute(s & 1);
        if (s + 1 < nk) sstore((s + 1) & 1);
        __syncthreads();
    }

    // Epilogue.  32x32 accumulator layout: lane holds column (lane & 31) and
    // rows (r/4)*8 + (lane/32)*4 + r%4 of its block, r = 0..15.
#pragma unroll
    for (int i = 0; i < S::MB; ++i) {
        if (i >= mact) continue;
        const int row_base = wm * S::WTM + 32 * i + (lane >> 5) * 4;
        if (GLU) {
#pragma unroll
            for (int j = 0; j < S::NBW / 2; ++j) {
                const int col = wn * (S::BN / 2 / S::WN) + 32 * j + (lane & 31);
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
                const int col = wn * (S::BN / S::WN) + 32 * j + (lane & 31);
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    out[(long)(row_base + (r >> 2) * 8 + (r & 3)) * ldo + col] = (uint16_t)f2bf_bits(acc[i][j][r]);
            }
        }
    }
}

}  // namespace moeapk
