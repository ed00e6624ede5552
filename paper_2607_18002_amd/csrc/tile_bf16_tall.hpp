// bf16 grouped-GEMM tile for tall row tiles (prefill), gfx950 MFMA
// v_mfma_f32_32x32x16_bf16.
//
// One 256-thread workgroup computes a BM x 256 output tile over the full K
// (BM = 192: 6 row blocks of 32).  Each wave owns 64 output columns for all
// BM rows: 6 row blocks x 2 column blocks of 32 x 32, 192 fp32 accumulators
// per lane.  Against the 128-row tile (tile_bf16.hpp) every weight fragment
// that streams into a wave's registers feeds 12 MFMAs instead of 8, so a
// workgroup pulls 1/3 fewer weight bytes through L1/L2 per flop.  That is
// what limits the 128-row tile inside the persistent kernel: only the few row
// tiles of one expert share a weight slice in an XCD's L2, and the tile's
// time grows with the number of distinct slices an XCD streams at once.
// (256 rows would fill all 256 AGPRs with accumulators; the register
// allocator then spills the operand registers, so 192 is the tallest tile.)
//  * B (weights, packed operand order) streams global -> registers through a
//    ring of D = 2 K steps (full tiles ran alike with D = 2..6; deeper rings
//    for short tiles made the mixed workload slower);
//  * A (activation rows, shared by the 4 waves) is loaded into registers one
//    K step ahead (AP = 2, two steps ahead, measured slower in situ) and
//    staged through double-buffered LDS (rows padded by 16 bytes: the
//    fragment reads are free of bank conflicts; a third stage, which lets a
//    step's first fragments be read before the barrier, also measured slower);
//  * A fragments are read from LDS two MFMA pairs ahead of their use.
// K order, GLU layout, row maps and the epilogue follow the 128-row tile; the
// epilogue runs in parts of at most 4 row blocks so its LDS staging stays at
// 72 KB.
#pragma once

#include "tile_bf16.hpp"

namespace moeapk {

// LDS bytes a tall tile needs: two A stages, or one epilogue part (128 rows)
// per wave.
template <class S>
struct TallLds {
    static constexpr int part = 4 * 128 * (S::WCOLS * 2 + 16);
    static constexpr int bytes = 2 * S::A_STAGE > part ? 2 * S::A_STAGE : part;
};

// One K step of MFMAs for MACT row blocks: the MFMA pair (i, j = 0..1) of
// K slice kk uses A fragment n = kk * MACT + i; fragment n + 2 is read from
// LDS while pair n issues (three fragment registers in rotation).
template <class S, int MACT>
__device__ __forceinline__ void mma_step_tall(f32x16 (&acc)[MACT][2], const bf16x8 (&rb)[2][4], const char* buf,
                                              int lane) {
    constexpr int NF = 4 * MACT;
    const char* arow = buf + (lane & 31) * S::LDS_ROW + (lane >> 5) * 64;   // lanes 32-63: +32 elements
    auto frag_addr = [&](int n) {
        const int kk = n / MACT, i = n % MACT;
        return arow + i * 32 * S::LDS_ROW + (kk >> 2) * 128 + (kk & 3) * 16;
    };
    bf16x8 af[3];
    af[0] = *(const bf16x8*)frag_addr(0);
    if (NF > 1) af[1] = *(const bf16x8*)frag_addr(1);
    __builtin_amdgcn_sched_group_barrier(0x100, NF > 1 ? 2 : 1, 0);
#pragma unroll
    for (int n = 0; n < NF; ++n) {
        const int kk = n / MACT, i = n % MACT;
        if (n + 2 < NF) af[(n + 2) % 3] = *(const bf16x8*)frag_addr(n + 2);
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[n % 3], rb[j][kk], acc[i][j], 0, 0, 0);
        if (n + 2 < NF) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
}

// Arguments as gemm_tile_bf16 (tile_bf16.hpp), with rows [0, 32*MACT) of a
// BM-row tile; weights must be packed (moe_pack_weights).
template <class S, bool GLU, int MACT, int D = 2, int AP = 1, class Hook = NoHook>
__device__ __forceinline__ void gemm_tile_tall(const uint16_t* __restrict__ A, int lda,
                                               const uint16_t* __restrict__ B, int ldb, int up_rows, int K,
                                               uint16_t* __restrict__ out, int ldo, char* lds,
                                               const int32_t* __restrict__ rowmap = nullptr, int k = 1,
                                               int a_rows = 0, Hook hook = Hook{}) {
    static_assert(MACT >= 1 && MACT <= S::MB && S::NBW == 2, "1..MB row blocks, 2 column blocks per wave");
    constexpr int CA = MACT * 32 / S::RPP;           // A chunks per thread and K step
    const int tid = threadIdx.x, lane = tid & 63, wn = tid >> 6;

    uint32_t boff[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        int row;
        if (GLU) row = wn * (S::WCOLS / 2) + (lane & 31) + (j == 0 ? 0 : up_rows);
        else row = wn * S::WCOLS + 32 * j + (lane & 31);
        boff[j] = (uint32_t)(row - (lane & 31)) * (uint32_t)ldb * 2u + (uint32_t)(lane * 16);
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
    const __amdgpu_buffer_rsrc_t Ab =
        make_rsrc(A, (uint32_t)(rowmap ? a_rows : MACT * 32) * (uint32_t)lda * 2u);
    const __amdgpu_buffer_rsrc_t Bb =
        make_rsrc(B, (uint32_t)(GLU ? up_rows + S::BN / 2 : S::BN) * (uint32_t)ldb * 2u);
    char* lds0 = lds;
    char* lds1 = lds + S::A_STAGE;

    f32x16 acc[MACT][2];
#pragma unroll
    for (int i = 0; i < MACT; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    u32x4 ra[AP][CA];                                 // A of steps s+1 .. s+AP (slot = step % AP)
    bf16x8 rb[D][2][4];                               // B of steps s .. s+D-1 (slot = step % D)
    const int nk = K / S::BK;                         // a multiple of D and of 2
    constexpr int KB = S::BK * 2;                     // bytes per K step of a row-major A row
    constexpr int KBB = S::BK * 64;                   // bytes per K step of a packed weight block
    static_assert(D % 2 == 0, "the LDS stages (step & 1) repeat within one pass of the B ring");
    static_assert(AP == 1 || AP == 2, "A is loaded one or two K steps ahead of its LDS store");

    // Branch-free K loop (loads past the last step are clamped to it), so the
    // compiler's wait counts stay exact.  A loads go before the B loads of the
    // same step, so waiting for A leaves later B loads in flight.
    const int last = nk - 1;
    load_a<CA>(ra[0], Ab, aoff, 0);
#pragma unroll
    for (int d = 0; d < D; ++d) load_b<S, true>(rb[d], Bb, boff, d * KBB);
    store_a<CA>(lds0, ra[0], alds);
#pragma unroll
    for (int j = 1; j <= AP; ++j) load_a<CA>(ra[j % AP], Ab, aoff, (j < last ? j : last) * KB);
    __syncthreads();
    for (int s0 = 0; s0 < nk; s0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            const int s = s0 + d;                     // s % AP == d % AP: D is even
            mma_step_tall<S, MACT>(acc, rb[d], (d & 1) ? lds1 : lds0, lane);
            store_a<CA>((d & 1) ? lds0 : lds1, ra[(d + 1) % AP], alds);
            const int sb = s + D < last ? s + D : last, sa = s + 1 + AP < last ? s + 1 + AP : last;
            load_a<CA>(ra[(d + 1) % AP], Ab, aoff, sa * KB);
            load_b<S, true>(rb[d], Bb, boff, sb * KBB);
            __syncthreads();
        }
    }
    hook();

    // Epilogue in parts of up to 4 row blocks: each wave stages its bf16
    // block in its own LDS region, reads it back row-wise and writes whole
    // 16-byte row chunks with device-coherent stores (sc1).
    constexpr int OC = GLU ? S::WCOLS / 2 : S::WCOLS;      // output columns per wave
    constexpr int ORB = OC * 2 + 16;                       // staged row pitch in bytes
    constexpr int HALF_STAGE = 128 * ORB;
    char* stg = lds + wn * HALF_STAGE;
    constexpr int CPO = OC * 2 / 16;                       // 16-byte chunks per output row
    constexpr int RPI = 64 / CPO;                          // rows per store instruction
    static_assert(64 % CPO == 0 && 32 % RPI == 0, "a store pass stays inside one 32-row block");
    const __amdgpu_buffer_rsrc_t Ob = make_rsrc(out, (uint32_t)(MACT * 32) * (uint32_t)ldo * 2u);
    const int orow = lane / CPO, och = lane % CPO;
    const uint32_t ooff = (uint32_t)orow * (uint32_t)ldo * 2u + (uint32_t)(wn * OC + och * 8) * 2u;
#pragma unroll
    for (int h = 0; h < (MACT + 3) / 4; ++h) {
        const int i0 = h * 4;
        const int nb_h = MACT - i0 < 4 ? MACT - i0 : 4;          // row blocks in this half (uniform)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            const int i = i0 + ii;
            if (i >= MACT) break;
            // one row block at a time: keeps the compiler from reading every
            // accumulator out of the AGPRs at once
            __builtin_amdgcn_sched_barrier(0);
            const int row_base = 32 * ii + (lane >> 5) * 4;
#pragma unroll
            for (int j = 0; j < OC / 32; ++j) {
                const int col = 32 * j + (lane & 31);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float v;
                    if (GLU) {
                        const float g = acc[i][0][r], u = acc[i][1][r];
                        v = g / (1.f + __expf(-g)) * u;
                    } else {
                        v = acc[i][j][r];
                    }
                    *(uint16_t*)(stg + (row_base + (r >> 2) * 8 + (r & 3)) * ORB + col * 2) = (uint16_t)f2bf_bits(v);
                }
            }
        }
#pragma unroll
        for (int p = 0; p < 4 * 32 / RPI; ++p) {
            if (p * RPI >= nb_h * 32) break;
            const u32x4 v = *(const u32x4_alias*)(stg + (p * RPI + orow) * ORB + och * 16);
            __builtin_amdgcn_raw_buffer_store_b128(
                v, Ob, (int)ooff, (int)((uint32_t)(i0 * 32 + p * RPI) * (uint32_t)ldo * 2u),
                GLU ? kStoreDevice : kStoreDeviceStream);
        }
        // A 16-byte store reads its data registers after it issues: two wait
        // states must pass before a VALU instruction overwrites them.  The next
        // part's first instructions are VALU work that may reuse those
        // registers, and the compiler does not insert the wait states across
        // the scheduling barrier that starts the part.
        if (h + 1 < (MACT + 3) / 4) asm volatile("s_nop 1");
    }
}

// Dispatch on the number of 32-row blocks holding valid rows (uniform per tile).
template <class S, bool GLU, class Hook = NoHook>
__device__ __forceinline__ void gemm_tile_tall_rows(int rows32, const uint16_t* A, int lda, const uint16_t* B,
                                                    int ldb, int up_rows, int K, uint16_t* out, int ldo, char* lds,
                                                    const int32_t* rowmap = nullptr, int k = 1, int a_rows = 0,
                                                    Hook hook = Hook{}) {
    static_assert(S::MB == 6, "dispatch written for 192-row tiles");
    switch (rows32 >> 5) {
        case 1: gemm_tile_tall<S, GLU, 1>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        case 2: gemm_tile_tall<S, GLU, 2>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        case 3: gemm_tile_tall<S, GLU, 3>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        case 4: gemm_tile_tall<S, GLU, 4>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        case 5: gemm_tile_tall<S, GLU, 5>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
        default: gemm_tile_tall<S, GLU, 6>(A, lda, B, ldb, up_rows, K, out, ldo, lds, rowmap, k, a_rows, hook); break;
    }
}

}  // namespace moeapk
