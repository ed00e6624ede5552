// bf16 grouped-GEMM tile on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// One 256-thread workgroup computes a BM x BN output tile over the full K.
// The four waves split the BN columns (BN/4 each) and all share the BM rows:
//  * B (weight rows, K-contiguous) is private to a wave, so it streams from
//    global memory straight into MFMA operand registers through a ring of
//    DEPTH K-step buffers (loads issued DEPTH steps ahead of their MFMAs), with
//    no LDS round trip.  Tiles with few valid rows do little MFMA work per K
//    step and have registers to spare, so they run a deeper ring: that is what
//    keeps enough weight bytes in flight to stream at HBM speed;
//  * A (activation rows, shared by the four waves) is loaded into registers
//    two K steps ahead and staged through double-buffered LDS, with rows padded
//    by 16 bytes so an operand read is free of bank conflicts.
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

// A tile calls hook() once, after its K loop and before its epilogue: the
// caller's chance to issue memory requests whose latency then overlaps the
// epilogue's stores (NoHook: nothing).
struct NoHook {
    __device__ __forceinline__ void operator()() const {}
};

// BAUX: cache policy of the weight loads (0, or kLoadStream).
template <int BM_, int BN_, int BK_, int BAUX_ = 0>
struct TileShape {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, BAUX = BAUX_;
    static constexpr int MB = BM / 32;               // 32-row blocks
    static constexpr int WCOLS = BN / 4;             // B rows (output columns) per wave
    static constexpr int NBW = WCOLS / 32;           // 32-column MFMA blocks per wave
    static constexpr int KK = BK / 16;               // MFMAs along K per K step
    static constexpr int LDS_ROW = BK * 2 + 16;      // bytes per LDS row of A
    static constexpr int A_STAGE = BM * LDS_ROW;
    // Epilogue staging: each wave's bf16 output block, rows padded by 16 bytes
    // (the widest case, WCOLS columns, is reserved for GLU tiles too).
    static constexpr int OUT_ROW = WCOLS * 2 + 16;
    static constexpr int OUT_STAGE = BM * OUT_ROW;
    static constexpr int LDS = 2 * A_STAGE > 4 * OUT_STAGE ? 2 * A_STAGE : 4 * OUT_STAGE;
    static constexpr int CPR = BK / 8;               // 16-byte chunks per A row and K step
    static constexpr int RPP = 256 / CPR;            // A rows loaded per pass of 256 threads
    static_assert(NBW >= 2 && NBW % 2 == 0, "GLU needs a gate and an up block per wave");
    static_assert(256 % CPR == 0 && RPP <= 32 && 32 % RPP == 0, "an A load pass stays inside one 32-row block");
};

template <class S, int MACT>
struct TileRegs {
    static constexpr int CA = MACT * 32 / S::RPP;    // A chunks per thread and K step
    // K steps of A and B in flight (both rings have this depth).  One step of
    // B takes NBW * KK * 4 registers and one of A CA * 4; the MFMA
    // accumulators take MACT * NBW * 16, so fewer valid rows leave room for
    // more steps (budget: 128 registers at 3-4 row blocks, 192 at 2, 256 at 1).
    static constexpr int B_STEP_REGS = S::NBW * S::KK * 4;
    static constexpr int B_BUDGET = MACT == 1 ? 256 : MACT == 2 ? 192 : 128;
    static constexpr int DEPTH_RAW = B_BUDGET / (B_STEP_REGS + CA * 4);
    static constexpr int DEPTH = DEPTH_RAW >= 8 ? 8 : DEPTH_RAW < 2 ? 2 : (DEPTH_RAW & ~1);
};

// Raw buffer loads: the tile's base address lives in an SGPR descriptor, the
// per-lane offset in one VGPR, the K-step offset in an SGPR and the per-MFMA
// offset in the instruction, so a load needs no address arithmetic.  The
// descriptor's size bounds the tile's extent (reads past it return zero).
constexpr int kBufferWord3 = 0x00020000;   // gfx9-family raw buffer: 32-bit data format, no swizzle
constexpr int kStoreDevice = 16;           // cache policy sc1: the store is coherent at device scope
constexpr int kLoadStream = 2;             // cache policy nt: data read once, the first to leave the L2
// sc1 + nt: GEMM-2 outputs (y_perm rows), read only by the combine, so they
// need not displace weight slices and activation rows from the L2
constexpr int kStoreDeviceStream = kStoreDevice | kLoadStream;

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
                B, (int)(boff[j] + (PACKED ? kk * 1024 : (kk >> 2) * 128 + (kk & 3) * 16)), k0b, S::BAUX);
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

// A   : tile row 0 at k = 0, row stride lda elements; rows [0, 32*MACT) are read.
//       With a row map (gathered operand): A is row 0 of a matrix of a_rows
//       rows, and tile row r is A's row rowmap[r] / k (rowmap[r] < 0: zero).
// B   : first B row of the tile (GLU: gate row n0), row stride ldb elements
// up_rows : GLU only, rows from the gate block to the matching up block (I)
// out : output tile origin, row stride ldo (bf16); rows [0, 32*MACT) written
template <class S, bool GLU, int MACT, bool PACKED = false, int D = TileRegs<S, MACT>::DEPTH,
          class Hook = NoHook>
__device__ __forceinline__ void gemm_tile_bf16(const uint16_t* __restrict__ A, int lda,
                                               const uint16_t* __restrict__ B, int ldb, int up_rows, int K,
                                               uint16_t* __restrict__ out, int ldo, char* lds,
                                               const int32_t* __restrict__ rowmap = nullptr, int k = 1,
                                               int a_rows = 0, Hook hook = Hook{}) {
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
        int src = r;
        if (rowmap) {
            const int a = rowmap[r];
            src = (a >= 0 && a / k < a_rows) ? a / k : -1;
        }
        // a gathered padding row gets an offset past the buffer's extent, which reads as zero
        aoff[i] = src >= 0 ? (uint32_t)src * (uint32_t)lda * 2u + c * 16 : 0x80000000u;
        alds[i] = r * S::LDS_ROW + c * 16;
    }
    // extents: A rows [0, 32*MACT) (gathered: [0, a_rows)); B rows [0, BN) or, for GLU,
    // gate rows [0, BN/2) and up rows [up_rows, up_rows + BN/2)
    const __amdgpu_buffer_rsrc_t Ab =
        make_rsrc(A, (uint32_t)(rowmap ? a_rows : MACT * 32) * (uint32_t)lda * 2u);
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

    u32x4 ra[D][CA];                                  // A of steps s+1 .. s+D (slot = step % D)
    bf16x8 rb[D][S::NBW][S::KK];                      // B of steps s .. s+D-1 (slot = step % D)
    const int nk = K / S::BK;                         // a multiple of D (see gemm_tile_bf16_rows)
    constexpr int KB = S::BK * 2;                     // bytes per K step of a row-major row
    constexpr int KBB = PACKED ? S::BK * 64 : KB;     // bytes per K step of a weight fragment stream
    static_assert(S::BK % 64 == 0, "K steps are whole 64-element chunks");
    static_assert(D % 2 == 0, "the LDS stages (step & 1) repeat within one pass of the ring");

    // The K loop has no branches: a step's loads are clamped to the last K
    // step instead of skipped (the spare loads are re-reads of data just
    // loaded, never consumed).  With no path-dependent loads the compiler's
    // wait counts stay exact.
    // vmcnt counts loads in issue order, so waiting for one load waits for
    // every load issued before it.  A runs as far ahead as B: step s stores
    // A of step s+1 into LDS and issues A of step s+1+D, then B of step s+D,
    // so A of step s+1 was issued right before B of step s (which step s
    // needs anyway) and waiting for it leaves B of steps s+1 .. s+D-1 in
    // flight.  (With A loaded two steps ahead and issued after B, that wait
    // also drained every B load older than two steps: the ring held about
    // two steps, whatever its depth.)  The prologue issues the same pairs.
    const int last = nk - 1;
    load_a<CA>(ra[0], Ab, aoff, 0);
#pragma unroll
    for (int y = 0; y + 1 < D; ++y) {
        load_a<CA>(ra[y + 1], Ab, aoff, (y + 1 < last ? y + 1 : last) * KB);
        __builtin_amdgcn_sched_barrier(0);
        load_b<S, PACKED>(rb[y], Bb, boff, y * KBB);
        __builtin_amdgcn_sched_barrier(0);
    }
    store_a<CA>(lds0, ra[0], alds);
    load_a<CA>(ra[0], Ab, aoff, (D < last ? D : last) * KB);
    __builtin_amdgcn_sched_barrier(0);
    load_b<S, PACKED>(rb[D - 1], Bb, boff, (D - 1) * KBB);
    __syncthreads();
    for (int s0 = 0; s0 < nk; s0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            const int s = s0 + d;                     // uniform; d and s & 1 are compile-time
            mma_step<S, MACT>(acc, rb[d], (d & 1) ? lds1 : lds0, lane);
            store_a<CA>((d & 1) ? lds0 : lds1, ra[(d + 1) % D], alds);
            const int sb = s + D < last ? s + D : last, sa = s + 1 + D < last ? s + 1 + D : last;
            load_a<CA>(ra[(d + 1) % D], Ab, aoff, sa * KB);
            __builtin_amdgcn_sched_barrier(0);
            load_b<S, PACKED>(rb[d], Bb, boff, sb * KBB);
            __syncthreads();
        }
    }
    hook();

    // Epilogue.  32x32 accumulator layout: lane holds column (lane & 31) and
    // rows (r/4)*8 + (lane/32)*4 + r%4 of its block, r = 0..15.  Each wave
    // writes its bf16 block into its own LDS region (the A stages are free: the
    // last K step ended with a barrier), reads it back row-wise and writes
    // whole 16-byte row chunks with device-coherent stores (sc1): the stores
    // reach the coherence point by themselves, so the tile needs no L2
    // write-back before it is committed.  A wave reads back only what it wrote
    // itself, and LDS keeps one wave's operations in order.
    constexpr int OC = GLU ? S::WCOLS / 2 : S::WCOLS;      // output columns per wave
    constexpr int ORB = OC * 2 + 16;                       // staged row pitch in bytes
    char* stg = lds + wn * S::OUT_STAGE;
#pragma unroll
    for (int i = 0; i < MACT; ++i) {
        const int row_base = 32 * i + (lane >> 5) * 4;
#pragma unroll
        for (int j = 0; j < OC / 32; ++j) {
            const int col = 32 * j + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float v;
                if (GLU) {
                    const float g = acc[i][j][r], u = acc[i][j + S::NBW / 2][r];
                    v = g / (1.f + __expf(-g)) * u;
                } else {
                    v = acc[i][j][r];
                }
                *(uint16_t*)(stg + (row_base + (r >> 2) * 8 + (r & 3)) * ORB + col * 2) = (uint16_t)f2bf_bits(v);
            }
        }
    }
    constexpr int CPO = OC * 2 / 16;                       // 16-byte chunks per output row
    constexpr int RPI = 64 / CPO;                          // rows per store instruction
    static_assert(64 % CPO == 0 && 32 % RPI == 0, "a store pass stays inside one 32-row block");
    const __amdgpu_buffer_rsrc_t Ob = make_rsrc(out, (uint32_t)(MACT * 32) * (uint32_t)ldo * 2u);
    const int orow = lane / CPO, och = lane % CPO;
    const uint32_t ooff = (uint32_t)orow * (uint32_t)ldo * 2u + (uint32_t)(wn * OC + och * 8) * 2u;
#pragma unroll
    for (int p = 0; p < MACT * 32 / RPI; ++p) {
        const u32x4 v = *(const u32x4_alias*)(stg + (p * RPI + orow) * ORB + och * 16);
        __builtin_amdgcn_raw_buffer_store_b128(v, Ob, (int)ooff, (int)((uint32_t)(p * RPI) * (uint32_t)ldo * 2u),
                                               GLU ? kStoreDevice : kStoreDeviceStream);
    }
}

// The K loop runs whole passes of the B ring: the ring depth for the tile's
// row count when it divides the number of K steps, else 2 (K is a multiple
// of 2 * BK).
template <class S, bool GLU, int MACT, bool PACKED, class Hook>
__device__ __forceinline__ void gemm_tile_bf16_depth(const uint16_t* A, int lda, const uint16_t* B, int ldb,
                                                     int up_rows, int K, uint16_t* out, int ldo, char* lds,
                                                     const int32_t* rowmap, int k, int a_rows, Hook hook) {
    constexpr int D = TileRegs<S, MACT>::DEPTH;
    if ((K / S::BK) % D == 0)
        gemm_tile_bf16<S, GLU, MACT, PACKED, D>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook);
    else
        gemm_tile_bf16<S, GLU, MACT, PACKED, 2>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook);
}

// Dispatch on the number of 32-row blocks holding valid rows (uniform per tile).
template <class S, bool GLU, bool PACKED, class Hook = NoHook>
__device__ __forceinline__ void gemm_tile_bf16_rows(int rows32, const uint16_t* A, int lda, const uint16_t* B, int ldb,
                                                    int up_rows, int K, uint16_t* out, int ldo, char* lds,
                                                    const int32_t* rowmap = nullptr, int k = 1, int a_rows = 0,
                                                    Hook hook = Hook{}) {
    static_assert(S::MB == 4, "dispatch written for 128-row tiles");
    switch (rows32 >> 5) {
        case 1: gemm_tile_bf16_depth<S, GLU, 1, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        case 2: gemm_tile_bf16_depth<S, GLU, 2, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        case 3: gemm_tile_bf16_depth<S, GLU, 3, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        default: gemm_tile_bf16_depth<S, GLU, 4, PACKED>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
    }
}

}  // namespace moeapk
