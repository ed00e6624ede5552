// fp8 (OCP E4M3FN) grouped-GEMM tile on gfx950 with fp32 block scales.
//
// Block-scaled product (weights in 128 x 128 blocks, activations in 1 x 128
// groups along K):
//   out[t][n] = sum_kb sx[t][kb] * sw[n/128][kb] * sum_{k in block kb} xq[t][k] * wq[n][k].
// The inner sum of each 128-element K block is two v_mfma_scale_f32_32x32x64_f8f6f4
// with unit E8M0 scales (127), i.e. a plain fp8 product accumulated in fp32,
// into a fresh accumulator; the block is then added to the running fp32 total
// with its two exact fp32 scales.  The scales are arbitrary fp32 values, which
// the MFMA's power-of-two block scales cannot express.
//
// Orientation: the MFMA's A operand is weight rows (output features) and its B
// operand is activation rows (tokens).  A lane's 32x32 accumulator then holds
// one token (column lane % 32) and 16 features of one 32-feature block, which
// all share one activation scale and one weight scale: folding a block into
// the total costs one multiply and 16 FMAs per lane.
//
// Workgroup: 4 waves; wave w owns features [w*WCOLS, (w+1)*WCOLS) (NBW blocks
// of 32) for all BM (up to 128) tokens.  Partial sums are kept for two row
// blocks at a time (one folds while the next one's MFMAs run), so the tile
// holds NBW * MACT running totals plus 2 * NBW partials: 192 accumulator
// registers at 128 tokens.  The taller the tile, the fewer weight bytes per
// flop it streams, and a 64-token tile was bound by that stream.  Weights stream global -> registers through a ring
// of DEPTH K steps (moe_pack_weights' fp8 layout: per 32-row block and 128-K
// chunk, [kk][half][lane][16 B]); activations are staged through double-
// buffered LDS (rows padded by 16 bytes); the tile's activation scales are
// staged in LDS once, as [K/128][BM].  MFMA K order: MFMA kk of a step covers
// elements kk*64 + (lane/32)*32 + [0, 32) of the block, in both operands.
#pragma once

#include "tile_bf16.hpp"

namespace moeapk {

// BAUX: cache policy of the weight loads (0, or kLoadStream).
template <int BM_, int BN_, int BAUX_ = 0>
struct TileShapeF8 {
    static constexpr int BM = BM_, BN = BN_, BK = 128, BAUX = BAUX_;
    static constexpr int MB = BM / 32;                // 32-token blocks
    static constexpr int WCOLS = BN / 4;              // features per wave
    static constexpr int NBW = WCOLS / 32;            // 32-feature blocks per wave
    static constexpr int KK = BK / 64;                // MFMAs along K per step
    static constexpr int LDS_ROW = BK + 16;           // bytes per staged activation row
    static constexpr int A_STAGE = BM * LDS_ROW;
    static constexpr int MAX_KB = 64;                 // K <= 8192
    static constexpr int SX_OFF = 2 * A_STAGE;        // activation scales [kb][BM] (f32)
    static constexpr int SX_BYTES = MAX_KB * BM * 4;
    static constexpr int H_ROW = (BN / 2) * 4 + 16;   // GLU epilogue: fp32 h row of BN/2 features
    static constexpr int OUT_ROW = WCOLS * 2 + 16;    // GEMM-2 epilogue: per-wave bf16 row
    static constexpr int EPI = BM * H_ROW > 4 * BM * OUT_ROW ? BM * H_ROW : 4 * BM * OUT_ROW;
    // weight scales of each wave's feature blocks, [wave][j][kb] (f32): read
    // from LDS in the K loop, since a global load there would be the youngest
    // in flight and waiting for it would drain the weight prefetch as well
    static constexpr int SW_OFF = SX_OFF + SX_BYTES;
    static constexpr int SW_BYTES = 4 * NBW * MAX_KB * 4;
    static constexpr int LDS = SW_OFF + SW_BYTES > EPI ? SW_OFF + SW_BYTES : EPI;
    static constexpr int CPR = BK / 16;               // 16-byte chunks per activation row and step
    static constexpr int RPP = 256 / CPR;             // activation rows per load pass
    static_assert(NBW == 2, "GLU pairs one gate and one up block per wave");
    static_assert(RPP <= 32 && 32 % RPP == 0, "a load pass stays inside one 32-row block");
};

template <class S, int MACT>
struct TileRegsF8 {
    static constexpr int CA = MACT * 32 / S::RPP;     // activation chunks per thread and step
    static constexpr int DEPTH = MACT == 1 ? 4 : 2;   // weight steps in flight (32 VGPRs each)
};

// Per-lane scale factors of one K step's block: the token's activation scale
// times each feature block's weight scale, folded into the running totals.
template <class S, int MACT>
__device__ __forceinline__ void fold_block(f32x16 (&tot)[S::NBW][MACT], const f32x16 (&part)[S::NBW], int i, float xs,
                                           const float (&cw)[S::NBW]) {
#pragma unroll
    for (int j = 0; j < S::NBW; ++j) {
        const float c = xs * cw[j];
#pragma unroll
        for (int r = 0; r < 16; ++r) tot[j][i][r] = __builtin_fmaf(part[j][r], c, tot[j][i][r]);
    }
}

// Weight operands of one K step: per block j and MFMA kk, 32 bytes per lane
// (two 16-byte halves, each a 1 KB contiguous wave load).
template <class S>
__device__ __forceinline__ void load_w8(i32x8 (&rw)[S::NBW][S::KK], __amdgpu_buffer_rsrc_t B,
                                        const uint32_t (&boff)[S::NBW], int k0b) {
#pragma unroll
    for (int j = 0; j < S::NBW; ++j)
#pragma unroll
        for (int kk = 0; kk < S::KK; ++kk) {
            const u32x4 lo = __builtin_amdgcn_raw_buffer_load_b128(B, (int)(boff[j] + kk * 2048), k0b, S::BAUX);
            const u32x4 hi = __builtin_amdgcn_raw_buffer_load_b128(B, (int)(boff[j] + kk * 2048 + 1024), k0b, S::BAUX);
            rw[j][kk] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
        }
}

// A   : activation codes of tile row 0, lda bytes per row; rows [0, 32*MACT) are read
// asc : activation scales of tile row 0 (f32), K/128 per row
// B   : packed weight codes, first row n0 of the tile (a multiple of 32);
//       GLU: gate rows n0 + [0, BN/2) and up rows n0 + up_rows + [0, BN/2)
// wsc : weight scales of the expert, [N/128][K/128]
// rowmap (optional, gathered operand): A and asc start at row 0 of a matrix of
//       a_rows rows; tile row r is its row rowmap[r] / k (rowmap[r] < 0: zero)
// GLU : out = h codes (ldo bytes per row), osc = h scales (ldsc floats per row);
//       else out = bf16 rows (ldo elements per row)
template <class S, bool GLU, int MACT, int D = TileRegsF8<S, MACT>::DEPTH, class Hook = NoHook>
__device__ __forceinline__ void gemm_tile_fp8(const uint8_t* __restrict__ A, int lda, const float* __restrict__ asc,
                                              const uint8_t* __restrict__ B, int n0, int up_rows,
                                              const float* __restrict__ wsc, int K, void* __restrict__ out, int ldo,
                                              float* __restrict__ osc, int ldsc, char* lds,
                                              const int32_t* __restrict__ rowmap = nullptr, int k = 1,
                                              int a_rows = 0, Hook hook = Hook{}) {
    constexpr int CA = TileRegsF8<S, MACT>::CA;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wn = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nkb = K / S::BK;

    // weight rows of this wave's feature blocks, and their scale rows
    uint32_t boff[S::NBW];
    const float* sw[S::NBW];
#pragma unroll
    for (int j = 0; j < S::NBW; ++j) {
        const int row = GLU ? (j == 0 ? 0 : up_rows) + wn * (S::WCOLS / 2) : wn * S::WCOLS + 32 * j;
        boff[j] = (uint32_t)row * (uint32_t)K + (uint32_t)(lane * 16);
        sw[j] = wsc + (long)((n0 + row) / 128) * nkb;
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
        aoff[i] = src >= 0 ? (uint32_t)src * (uint32_t)lda + c * 16 : 0x80000000u;
        alds[i] = r * S::LDS_ROW + c * 16;
    }
    const __amdgpu_buffer_rsrc_t Ab = make_rsrc(A, (uint32_t)(rowmap ? a_rows : MACT * 32) * (uint32_t)lda);
    const __amdgpu_buffer_rsrc_t Bb =
        make_rsrc(B, (uint32_t)(GLU ? up_rows + S::BN / 2 : S::BN) * (uint32_t)K);
    char* lds0 = lds;
    char* lds1 = lds + S::A_STAGE;
    float* sx = (float*)(lds + S::SX_OFF);

    // this wave's weight scale rows, then the tile's activation scales
    // transposed to [kb][token]
    float* swl = (float*)(lds + S::SW_OFF) + wn * (S::NBW * S::MAX_KB);
    for (int idx = lane; idx < S::NBW * nkb; idx += 64) {
        const int j = idx / nkb, kb = idx - j * nkb;
        swl[j * S::MAX_KB + kb] = sw[j][kb];
    }
    for (int idx = tid; idx < MACT * 32 * nkb; idx += 256) {
        const int r = idx / nkb, kb = idx - r * nkb;
        int src = r;
        if (rowmap) {
            const int a = rowmap[r];
            src = (a >= 0 && a / k < a_rows) ? a / k : -1;
        }
        sx[kb * S::BM + r] = src >= 0 ? asc[(long)src * nkb + kb] : 0.f;
    }

    f32x16 tot[S::NBW][MACT];
#pragma unroll
    for (int j = 0; j < S::NBW; ++j)
#pragma unroll
        for (int i = 0; i < MACT; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) tot[j][i][r] = 0.f;

    u32x4 ra[CA];
    i32x8 rw[D][S::NBW][S::KK];
    const int arow = (lane & 31) * S::LDS_ROW + (lane >> 5) * 32;      // lanes 32-63: +32 bytes
    constexpr int KBW = 32 * S::BK;                                   // bytes per K step of a 32-row block

    // Branch-free K loop (K/128 is a multiple of D): loads are clamped to the
    // last step instead of skipped, so the compiler's wait counts stay exact
    // and a step's waits leave the later steps' weight loads in flight.
    // In every step the next step's A loads are issued before this step's
    // weight loads, so waiting for A leaves those weights in flight; the
    // prologue keeps that order too (the last weight step after A of step 1),
    // since the loop's wait counts hold for its entry as well.
    const int last = nkb - 1;
#pragma unroll
    for (int d = 0; d + 1 < D; ++d) load_w8<S>(rw[d], Bb, boff, d * KBW);
    load_a<CA>(ra, Ab, aoff, 0);
    store_a<CA>(lds0, ra, alds);
    load_a<CA>(ra, Ab, aoff, (1 < last ? 1 : last) * S::BK);
    __builtin_amdgcn_sched_barrier(0);                 // keep the issue order
    load_w8<S>(rw[D - 1], Bb, boff, (D - 1) * KBW);
    __syncthreads();
    for (int s0 = 0; s0 < nkb; s0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            const int s = s0 + d;                                      // uniform; d and s & 1 are compile-time
            const char* cur = (d & 1) ? lds1 : lds0;
            float cw[S::NBW];
#pragma unroll
            for (int j = 0; j < S::NBW; ++j) cw[j] = swl[j * S::MAX_KB + s];
            const float* sxs = sx + s * S::BM + (lane & 31);
            // Row block by row block: the block's two MFMAs per feature block
            // go into a fresh partial (two partial sets alternate), and the
            // previous row block's partial is folded into its total while
            // they run, so partials take 2 * NBW accumulators, not MACT * NBW.
            auto frag = [&](int i, int kk) {
                const char* p = cur + arow + i * 32 * S::LDS_ROW + kk * 64;
                const u32x4 lo = *(const u32x4_alias*)p, hi = *(const u32x4_alias*)(p + 16);
                return i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
            };
            f32x16 part[2][S::NBW];
            i32x8 xa[2][S::KK];
#pragma unroll
            for (int kk = 0; kk < S::KK; ++kk) xa[0][kk] = frag(0, kk);
#pragma unroll
            for (int i = 0; i < MACT; ++i) {
                if (i + 1 < MACT) {
#pragma unroll
                    for (int kk = 0; kk < S::KK; ++kk) xa[(i + 1) & 1][kk] = frag(i + 1, kk);
                }
#pragma unroll
                for (int j = 0; j < S::NBW; ++j) {
                    const f32x16 c0 = {};
#pragma unroll
                    for (int kk = 0; kk < S::KK; ++kk)
                        part[i & 1][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                            rw[d][j][kk], xa[i & 1][kk], kk == 0 ? c0 : part[i & 1][j], 0, 0, 0, 127, 0, 127);
                }
                if (i > 0) fold_block<S, MACT>(tot, part[(i - 1) & 1], i - 1, sxs[32 * (i - 1)], cw);
            }
            store_a<CA>((d & 1) ? lds0 : lds1, ra, alds);
            const int sw_ = s + D < last ? s + D : last, sa = s + 2 < last ? s + 2 : last;
            load_a<CA>(ra, Ab, aoff, sa * S::BK);
            __builtin_amdgcn_sched_barrier(0);
            load_w8<S>(rw[d], Bb, boff, sw_ * KBW);
            fold_block<S, MACT>(tot, part[(MACT - 1) & 1], MACT - 1, sxs[32 * (MACT - 1)], cw);
            __syncthreads();
        }
    }
    hook();

    // Accumulator layout: lane holds token 32*i + (lane & 31) and features
    // 32*j + (r/4)*8 + (lane/32)*4 + r%4 of its wave's columns, r = 0..15.
    if (GLU) {
        // h = silu(g) * u in fp32 -> LDS [token][BN/2]; then each token row's
        // BN/2 = 128 values (one scale group) are quantized with
        // scale = max(amax, 1e-4) / 448, clamped to +-448 before the convert
        // (the hardware convert does not saturate).
        static_assert(S::BN / 2 == 128, "one h scale group per GEMM-1 tile");
        char* hb = lds;
#pragma unroll
        for (int i = 0; i < MACT; ++i) {
            const int t = 32 * i + (lane & 31);
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                f32x4 v;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float gt = tot[0][i][g * 4 + q], up = tot[1][i][g * 4 + q];
                    v[q] = gt / (1.f + __expf(-gt)) * up;
                }
                *(f32x4*)(hb + t * S::H_ROW + (wn * 32 + g * 8 + (lane >> 5) * 4) * 4) = v;
            }
        }
        __syncthreads();
        const int qq = tid & 3;                                     // 4 threads per token row, 32 values each
        for (int t = tid >> 2; t < MACT * 32; t += 64) {
            const f32x4* src = (const f32x4*)(hb + t * S::H_ROW + qq * 128);
            f32x4 v[8];
            float amax = 0.f;
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                v[k] = src[k];
#pragma unroll
                for (int q = 0; q < 4; ++q) amax = fmaxf(amax, fabsf(v[k][q]));
            }
            amax = fmaxf(amax, __shfl_xor(amax, 1, 64));
            amax = fmaxf(amax, __shfl_xor(amax, 2, 64));
            const float m = fmaxf(amax, 1e-4f);
            const float inv = 448.f / m;
            u32x4 code[2];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                float c4[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) c4[q] = fminf(fmaxf(v[k][q] * inv, -448.f), 448.f);
                int w = __builtin_amdgcn_cvt_pk_fp8_f32(c4[0], c4[1], 0, false);
                w = __builtin_amdgcn_cvt_pk_fp8_f32(c4[2], c4[3], w, true);
                code[k >> 2][k & 3] = (uint32_t)w;
            }
            const __amdgpu_buffer_rsrc_t Ob = make_rsrc(out, (uint32_t)(MACT * 32) * (uint32_t)ldo);
            const int o = t * ldo + qq * 32;
            __builtin_amdgcn_raw_buffer_store_b128(code[0], Ob, o, 0, kStoreDevice);
            __builtin_amdgcn_raw_buffer_store_b128(code[1], Ob, o + 16, 0, kStoreDevice);
            if (qq == 0) __hip_atomic_store(osc + (long)t * ldsc, m / 448.f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    } else {
        // bf16 rows through per-wave LDS staging, written as 16-byte row chunks
        char* stg = lds + wn * (S::BM * S::OUT_ROW);
#pragma unroll
        for (int i = 0; i < MACT; ++i) {
            const int t = 32 * i + (lane & 31);
#pragma unroll
            for (int j = 0; j < S::NBW; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const uint32_t p0 = f2bf_bits(tot[j][i][g * 4 + 0]) | (f2bf_bits(tot[j][i][g * 4 + 1]) << 16);
                    const uint32_t p1 = f2bf_bits(tot[j][i][g * 4 + 2]) | (f2bf_bits(tot[j][i][g * 4 + 3]) << 16);
                    *(u32x2*)(stg + t * S::OUT_ROW + (32 * j + g * 8 + (lane >> 5) * 4) * 2) = u32x2{p0, p1};
                }
        }
        constexpr int CPO = S::WCOLS * 2 / 16;                     // 16-byte chunks per staged row
        constexpr int RPI = 64 / CPO;                              // rows per store instruction
        const __amdgpu_buffer_rsrc_t Ob = make_rsrc(out, (uint32_t)(MACT * 32) * (uint32_t)ldo * 2u);
        const int orow = lane / CPO, och = lane % CPO;
        const uint32_t ooff = (uint32_t)orow * (uint32_t)ldo * 2u + (uint32_t)(wn * S::WCOLS + och * 8) * 2u;
#pragma unroll
        for (int p = 0; p < MACT * 32 / RPI; ++p) {
            const u32x4 v = *(const u32x4_alias*)(stg + (p * RPI + orow) * S::OUT_ROW + och * 16);
            __builtin_amdgcn_raw_buffer_store_b128(v, Ob, (int)ooff, (int)((uint32_t)(p * RPI) * (uint32_t)ldo * 2u),
                                                   kStoreDeviceStream);
        }
    }
}

// The K loop runs whole passes of the weight ring: the ring depth for the
// tile's row count when it divides K/128, else 2 (K is a multiple of 256).
template <class S, bool GLU, int MACT, class Hook>
__device__ __forceinline__ void gemm_tile_fp8_depth(const uint8_t* A, int lda, const float* asc, const uint8_t* B,
                                                    int n0, int up_rows, const float* wsc, int K, void* out, int ldo,
                                                    float* osc, int ldsc, char* lds, const int32_t* rowmap,
                                                    int k, int a_rows, Hook hook) {
    constexpr int D = TileRegsF8<S, MACT>::DEPTH;
    if ((K / S::BK) % D == 0)
        gemm_tile_fp8<S, GLU, MACT, D>(A, lda, asc, B, n0, up_rows, wsc, K, out, ldo, osc, ldsc, lds, rowmap, k,
                                       a_rows, hook);
    else
        gemm_tile_fp8<S, GLU, MACT, 2>(A, lda, asc, B, n0, up_rows, wsc, K, out, ldo, osc, ldsc, lds, rowmap, k,
                                       a_rows, hook);
}

template <class S, bool GLU, class Hook = NoHook>
__device__ __forceinline__ void gemm_tile_fp8_rows(int rows32, const uint8_t* A, int lda, const float* asc,
                                                   const uint8_t* B, int n0, int up_rows, const float* wsc, int K,
                                                   void* out, int ldo, float* osc, int ldsc, char* lds,
                                                   const int32_t* rowmap = nullptr, int k = 1, int a_rows = 0,
                                                   Hook hook = Hook{}) {
    static_assert(S::MB == 4, "dispatch written for 128-row tiles");
    switch (rows32 >> 5) {
        case 1: gemm_tile_fp8_depth<S, GLU, 1>(A, lda, asc, B, n0, up_rows, wsc, K, out, ldo, osc, ldsc, lds, rowmap,
                                               k, a_rows, hook); break;
        case 2: gemm_tile_fp8_depth<S, GLU, 2>(A, lda, asc, B, n0, up_rows, wsc, K, out, ldo, osc, ldsc, lds, rowmap,
                                               k, a_rows, hook); break;
        case 3: gemm_tile_fp8_depth<S, GLU, 3>(A, lda, asc, B, n0, up_rows, wsc, K, out, ldo, osc, ldsc, lds, rowmap,
                                               k, a_rows, hook); break;
        default: gemm_tile_fp8_depth<S, GLU, 4>(A, lda, asc, B, n0, up_rows, wsc, K, out, ldo, osc, ldsc, lds, rowmap,
                                                k, a_rows, hook); break;
    }
}

}  // namespace moeapk
