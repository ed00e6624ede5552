/*
 * moe_apk.h -- C ABI of the MI355X (gfx950) routed-expert MoE hot path.
 *
 * One GPU's share of a routed-expert MoE layer whose prefill and decode tokens
 * share the same local experts (ExpertPlex: Overview; Adaptive Persistent
 * Kernel; Evaluation "Implementation"):
 *
 *   moe_topk_route              top-k softmax gating                (step a1)
 *   moe_permute                 per-expert contiguous layout        (step a2)
 *   moe_grouped_ffn_persistent  SwiGLU expert FFN as one persistent
 *                               kernel with a device tile scheduler (steps a3-a6)
 *   moe_combine                 weighted combine to token order     (step a7)
 *
 * Conventions (all calls):
 *  - Pointers are DEVICE pointers unless marked "host".  The caller owns every
 *    buffer; no call allocates device memory.  Scratch space is a
 *    caller-allocated workspace whose size is returned by a *_workspace_bytes
 *    query.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *    stream) and never synchronise.
 *  - Argument errors are detected on the host before anything is launched and
 *    returned as a negative moe_status_t; moe_last_error() then holds a
 *    message (thread-local).
 *  - Data-dependent errors (an expert id out of range, a capacity overflow, a
 *    bounded wait that timed out, an abort) are written by the kernels to the
 *    caller's device status word (first error wins); kernels never write out
 *    of bounds because of them.  The caller reads the word when it next
 *    synchronises.
 *  - No C++ exception crosses this interface.
 *  - Supported device: gfx950 only (MOE_ERR_UNSUPPORTED elsewhere).
 */
#ifndef MOE_APK_H
#define MOE_APK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t moe_status_t;
#define MOE_OK               0
#define MOE_ERR_INVALID_ARG (-1) /* null pointer, bad size, inconsistent descriptor            */
#define MOE_ERR_UNSUPPORTED (-2) /* dtype / shape / device not supported by the kernels        */
#define MOE_ERR_CAPACITY    (-3) /* buffer capacity below the maximum routed volume            */
#define MOE_ERR_HIP         (-4) /* a HIP runtime call or kernel launch failed                 */
#define MOE_ERR_ABORTED     (-5) /* device: the abort word was set                             */
#define MOE_ERR_TIMEOUT     (-6) /* device: a bounded wait exceeded its spin limit             */
#define MOE_ERR_BAD_EXPERT  (-7) /* device: an expert id outside [-1, E_local)                 */
#define MOE_ERR_INTERNAL    (-8) /* device: a scheduler invariant failed; the kernel stopped
                                    before touching memory outside the op's buffers         */

typedef int32_t moe_dtype_t;
#define MOE_F32      0
#define MOE_BF16     1
#define MOE_FP8_E4M3 2   /* OCP E4M3FN, max 448, no infinities */

typedef int32_t moe_phase_t;
#define MOE_PREFILL 0
#define MOE_DECODE  1

#define MOE_MAX_OPS 16   /* operations per persistent launch */

typedef int32_t moe_layout_t;
#define MOE_LAYOUT_ROWMAJOR 0   /* [E, N, K], K contiguous                        */
#define MOE_LAYOUT_PACKED   1   /* written by moe_pack_weights (see below)        */

/* ------------------------------------------------------------------------- a1
 * Top-k gating (Background, "MoE LLM Inference": the router selects a top-k
 * subset of routed experts per token).  Reading taken for the unspecified
 * gating function: softmax over the k largest fp32 logits (equal to softmax
 * over all experts, select, renormalise), slots in descending-logit order,
 * equal logits (including -0.0 and +0.0) to the lower expert index.
 *
 *  logits    [T, E_global] f32, row-major; must be finite (NaN/inf give
 *            unspecified ids and weights, never out-of-bounds writes)
 *  topk_ids  [T, top_k] i32 out: local id (global id - local_begin) when the
 *            expert lies in [local_begin, local_begin + E_local), else -1
 *  topk_w    [T, top_k] f32 out: renormalised weights over all k slots
 *            (non-local slots keep their weight; the other expert-parallel
 *            ranks hold the rest of the sum)
 * Limits: 1 <= E_global <= 1024, 1 <= top_k <= min(E_global, 32), T >= 0
 * (T == 0 launches nothing), 0 <= local_begin, E_local >= 1.
 */
moe_status_t moe_topk_route(const float* logits, int32_t T, int32_t E_global, int32_t top_k,
                            int32_t local_begin, int32_t E_local,
                            int32_t* topk_ids, float* topk_w, void* stream);

/* The same gating for up to MOE_MAX_OPS operations (e.g. the layers and
 * phases of one persistent launch) in ONE kernel launch: each entry is one
 * moe_topk_route call's arguments, with the same meaning, limits and results
 * (bitwise).  ops: host array of n_ops entries, read before the call returns;
 * argument errors of any entry are returned before anything is launched. */
typedef struct moe_route_args {
    const float* logits;
    int32_t T, E_global, top_k, local_begin, E_local;
    int32_t* topk_ids;
    float* topk_w;
    /* Masked layout (the decode layout of "Prefill-Decode Disaggregation":
     * a fixed region of `slots` rows per local expert and a per-expert count,
     * filled as routing decides, with no packing pass).  With counts non-NULL
     * the entry also places every local slot a = t*top_k + j of expert e at
     * row e*slots + (the number of assignments a' < a of expert e), so the
     * rows of a region are its assignments in ascending a (deterministic,
     * bit-exact), and writes assign_to_row[a] (-1 for a slot that is not
     * local), row_to_assign[row] and counts[e] (no zeroing needed before).
     * The FFN then takes counts, offsets[e] = e*slots (offsets[E_local] =
     * E_local*slots) and capacity E_local*slots; moe_permute is not called.
     * Rows of a region past its count keep stale row_to_assign entries; the
     * FFN's gather bounds every entry by T*top_k and their outputs are never
     * read.
     *  slots     a multiple of 32, >= T (a token has at most one slot per expert)
     *  place_ws  moe_route_place_workspace_bytes(T, E_local) bytes of device
     *            memory, 8-byte aligned, zero before its first use (allocate
     *            it zeroed); the call leaves it ready for the next call with
     *            the same or a smaller T.  Calls that share it must not
     *            overlap in time.  (Routing blocks of a masked entry take
     *            chunks of 4 tokens up to 2048 tokens, of 16 above.)
     *  error_flag NULL or a device i32 status word: MOE_ERR_INTERNAL if
     *            place_ws was not zero before its first use, MOE_ERR_TIMEOUT
     *            if a wait for another block's counts exceeded its bound
     * Limits: 1 <= T < 2^29, E_local <= 1024, top_k <= 32.
     * With counts NULL the remaining fields are ignored. */
    int32_t slots, pad0;
    int32_t* counts;
    void* place_ws;
    int32_t* assign_to_row;
    int32_t* row_to_assign;
    int32_t* error_flag;
} moe_route_args;
moe_status_t moe_topk_route_batch(const moe_route_args* ops, int32_t n_ops, void* stream);
/* Bytes of place_ws a masked entry with T tokens and E_local experts needs
 * (0 if T < 1 or E_local < 1). */
size_t moe_route_place_workspace_bytes(int32_t T, int32_t E_local);

/* ------------------------------------------------------------------------- a2
 * Permutation into per-expert contiguous segments at final offsets
 * (Background, "Prefill-Decode Disaggregation": the contiguous layout;
 * "One-Sided Dispatch and Combine": routing fixes each expert's destination
 * and final offset before activations are written, into buffers sized for
 * the maximum routed volume).
 *
 * Assignment a = t*top_k + j.  Expert e's segment starts at offsets[e], a
 * multiple of row_align; its rows are e's assignments in ascending a
 * (deterministic, bit-exact); the segment is padded to a multiple of
 * row_align with rows whose row_to_assign is -1 and whose x_perm row is zero.
 *
 *  topk_ids       [T, top_k] i32 (from moe_topk_route); ids outside
 *                 [-1, E_local) set MOE_ERR_BAD_EXPERT and are treated as -1
 *  x              [T, H] activations: bf16, or fp8 codes with
 *  x_scales       [T, H/128] f32 per-row group scales (fp8 only, else NULL)
 *  row_align      segment alignment the FFN op that consumes the layout
 *                 needs (moe_ffn_row_align()); 1 <= row_align <= 1024
 *  capacity       rows of row_to_assign / x_perm; must be at least
 *                 T*min(top_k, E_local) + E_local*(row_align-1)
 *  counts         [E_local] i32 out     offsets [E_local+1] i32 out
 *  row_to_assign  [capacity] i32 out (rows >= offsets[E_local] untouched)
 *  assign_to_row  [T*top_k] i32 out (-1 for non-local slots)
 *  x_perm         [capacity, H] out, same dtype as x (rows >= offsets[E_local]
 *                 untouched);  x_perm_scales [capacity, H/128] f32 out (fp8).
 *                 x_perm NULL: only the maps are built (padding rows of
 *                 row_to_assign still set to -1); x and x_scales may then be
 *                 NULL -- the FFN gathers its rows from x itself (moe_op_desc.x)
 *  workspace      moe_permute_workspace_bytes(T, top_k, E_local) bytes of
 *                 device memory, zero before its first use (allocate it
 *                 zeroed); every call leaves its first 256 bytes zero again.
 *                 Calls that share a workspace must not overlap in time.
 *  error_flag     device i32 status word (data errors; not cleared here)
 * Limits: 1 <= E_local <= 1024, H a multiple of 128.
 */
size_t moe_permute_workspace_bytes(int32_t T, int32_t top_k, int32_t E_local);
moe_status_t moe_permute(const int32_t* topk_ids, int32_t T, int32_t top_k, int32_t E_local,
                         const void* x, moe_dtype_t x_dtype, const float* x_scales, int32_t H,
                         int32_t row_align, int32_t capacity,
                         int32_t* counts, int32_t* offsets, int32_t* row_to_assign,
                         int32_t* assign_to_row, void* x_perm, float* x_perm_scales,
                         void* workspace, int32_t* error_flag, void* stream);

/* The same permutation for up to MOE_MAX_OPS operations with one launch per
 * pass (count, scatter; the optional activation copies stay one launch per
 * op): each entry is one moe_permute call's arguments, same meaning, limits
 * and results (bitwise).  Entries must not share a workspace.  ops: host
 * array of n_ops entries, read before the call returns; argument errors of
 * any entry are returned before anything is launched. */
typedef struct moe_permute_args {
    const int32_t* topk_ids;
    int32_t T, top_k, E_local;
    moe_dtype_t x_dtype;
    const void* x;
    const float* x_scales;
    int32_t H, row_align, capacity, pad0;
    int32_t* counts;
    int32_t* offsets;
    int32_t* row_to_assign;
    int32_t* assign_to_row;
    void* x_perm;
    float* x_perm_scales;
    void* workspace;
    int32_t* error_flag;
} moe_permute_args;
moe_status_t moe_permute_batch(const moe_permute_args* ops, int32_t n_ops, void* stream);

/* ------------------------------------------------------------------------- a3-a6
 * Operation template (Adaptive Persistent Kernel, "Tile-Level Scheduling":
 * buffers and descriptors of every MoE operation are built before the
 * persistent kernel starts; at run time a ready signal instantiates the
 * operation into the decode or prefill queue).
 *
 * The op computes, for every local expert e and each of its rows r,
 *   h[r]      = silu(x_perm[r] . Wg_e^T) * (x_perm[r] . Wu_e^T)     (GEMM-1 + activation)
 *   y_perm[r] = h[r] . Wd_e^T                                        (GEMM-2)
 * with fp32 accumulation.  bf16 ops round h to bf16; fp8 ops quantize h per
 * row per 128 columns (scale = max(amax, 1e-4)/448, round to nearest even,
 * clamped to +-448).  y_perm rows of padding (row >= count within a segment)
 * are either zero or left untouched; they are never combined.
 */
typedef struct moe_op_desc {
    int32_t phase;            /* MOE_PREFILL or MOE_DECODE                              */
    int32_t layer;            /* informational; recorded in the trace                   */
    int32_t E_local, H, I;    /* H, I multiples of 256                                  */
    int32_t capacity;         /* rows of x_perm / h / y_perm                            */
    int32_t row_align;        /* must equal moe_ffn_row_align(phase, dtype)             */
    moe_dtype_t dtype;        /* MOE_BF16 or MOE_FP8_E4M3 (activations and weights)      */
    const int32_t* counts;    /* [E_local]     from moe_permute                          */
    const int32_t* offsets;   /* [E_local+1]   from moe_permute                          */
    const void*  x_perm;      /* [capacity, H]                                          */
    const float* x_perm_scales;      /* [capacity, H/128]            fp8 only           */
    const void*  w_gate_up;          /* [E_local, 2I, H] gate rows 0..I-1, up rows I..2I-1 */
    const float* w_gate_up_scales;   /* [E_local, 2I/128, H/128]     fp8 only           */
    const void*  w_down;             /* [E_local, H, I]                                  */
    const float* w_down_scales;      /* [E_local, H/128, I/128]      fp8 only           */
    void*  h;                 /* [capacity, I] intermediate (bf16, or fp8 codes)         */
    float* h_scales;          /* [capacity, I/128]              fp8 only                 */
    void*  y_perm;            /* [capacity, H] bf16 out                                  */
    /* Readiness ("One-Sided Dispatch and Combine": a ready signal is published
     * only after the payload is visible).  The op is ready when ALL hold:   */
    const uint32_t* release_word; /* NULL, or *release_word != 0 (system-scope acquire) */
    int64_t release_after_ns;     /* < 0: no time condition; else device wall clock >=
                                     kernel start + release_after_ns                     */
    int32_t depends_on_op;        /* -1, or an EARLIER op index that must be done...     */
                                  /* (an order of start times: an op's inputs are ready
                                     when the launch starts or when its release word is
                                     set, never outputs of another op of the launch)    */
    moe_layout_t weight_layout;   /* layout of w_gate_up / w_down: MOE_LAYOUT_PACKED      */
    int64_t gap_ns;               /* ...for at least gap_ns                              */
    uint32_t* done_word;          /* NULL, or set to 1 (system-scope release) when the
                                     op's last tile has committed                        */
    /* Fused gather (Evaluation, "Implementation": the MoE data pre-processing
     * fused into the persistent kernel).  With x_perm NULL and x set, GEMM-1
     * reads row r of a segment straight from x[row_to_assign[r] / top_k]
     * (padding rows, row_to_assign -1, read as zero) and, for fp8, its scales
     * from x_scales; moe_permute then only builds the maps (x_perm NULL).   */
    const void*  x;               /* [T, H] activations (bf16 or fp8 codes), or NULL    */
    const float* x_scales;        /* [T, H/128]                   fp8 only            */
    const int32_t* row_to_assign; /* [capacity] from moe_permute                       */
    int32_t T, top_k;             /* tokens (rows of x); slots per token                */
    /* Fused combine (Adaptive Persistent Kernel; Evaluation, "Implementation":
     * the MoE data post-processing fused into the persistent kernel).  With y
     * set, once every GEMM tile of the op has committed the kernel runs the
     * op's combine tiles (32 tokens each): y[t] = sum over the token's local
     * slots j, ascending, of topk_w[t,j] * y_perm[assign_to_row[t*top_k+j]],
     * accumulated in fp32 exactly as moe_combine does (so the two agree bit for
     * bit); tokens with no local slot get zeros.  The op completes (done word,
     * dependants, t_done) only after its combine tiles.  y is written with
     * device-coherent stores.  An assign_to_row entry >= capacity sets
     * MOE_ERR_INTERNAL and is skipped.  With y NULL the caller runs
     * moe_combine after the launch.                                            */
    const int32_t* assign_to_row; /* [T*top_k] from moe_permute (-1: slot not local)  */
    const float* topk_w;          /* [T, top_k] from moe_topk_route                   */
    void* y;                      /* [T, H] out, or NULL                              */
    moe_dtype_t y_dtype;          /* MOE_BF16 or MOE_F32                              */
    int32_t reserved_c;           /* 0                                                 */
} moe_op_desc;

/* Per-tile trace record (times in device wall-clock ticks, 100 MHz on gfx950).
 * A tile's life: the scheduling step that picked it began at t_boundary (it
 * first committed the workgroup's previous tile), its polls of the scheduler
 * words had returned at t_polled, the tile was claimed at t_claim, its
 * dependencies were met at t_start, and its outputs were committed at t_end.
 * c_start / c_end: the shader clock counter (s_memtime) at t_start / t_end, so
 * (c_end - c_start) / (t_end - t_start) is the clock the tile ran at. */
typedef struct moe_trace_rec {
    int16_t op, stage;        /* stage 1 = GEMM-1 (+activation), 2 = GEMM-2, 3 = combine */
    int16_t wg, xcc;          /* workgroup index and the XCD it ran on                  */
    int32_t expert, mblk;     /* local expert and row tile within its segment          */
    int16_t nblk, rows;       /* column block and valid rows in the tile               */
    /* The inputs of the decision that picked the tile: the quota q' it used,
     * which phases had claimable work in its polls (bit 0 decode, bit 1
     * prefill), and how it was taken: 0 from the workgroup's preferred phase,
     * 1 from the other phase (the preferred phase had no tile left to claim),
     * 2 claimed ahead during the previous tile, 3 a combine tile.           */
    int16_t quota_seen;
    uint8_t phases_seen, how;
    uint64_t t_boundary, t_polled, t_claim, t_start, t_end;
    uint64_t c_start, c_end;
} moe_trace_rec;

/* Per-op statistics written by the persistent kernel (times in wall-clock ticks). */
typedef struct moe_op_stats {
    uint64_t t_seen;          /* the ready signal was observed (at a tile boundary)    */
    uint64_t t_ready;         /* instantiation done: the op's tiles became claimable    */
    uint64_t t_first;         /* first tile started                                     */
    uint64_t t_done;          /* op finished: its last tile (combine tile, if fused) committed */
    int32_t x_moe;            /* Eq. (3) footprint: row tiles at the class's tile height */
    int32_t n_tiles;          /* GEMM-1 + GEMM-2 tiles (+ combine tiles, if fused)       */
    int32_t quota;            /* decode ops: q' of Eq. (4) in workgroups; prefill: 0    */
    int32_t reserved;
} moe_op_stats;

/* Scheduler policy ("Online SM Reallocation", Eq. (4)): under contention decode
 * may hold up to q' = min(Q_max, ceil_c(q * x_moe / x*_moe)) workgroups and
 * prefill takes the rest; a lone ready phase takes every workgroup.  Workgroups
 * with index < q' prefer decode tiles, the others prefer prefill; any
 * workgroup takes the other phase's tile when its preferred queue is empty;
 * a workgroup switches phase only between tiles. */
typedef struct moe_sched_config {
    int32_t n_workgroups;     /* 0 = one per CU                                         */
    int32_t decode_quota_wg;  /* q  (e.g. 64 = 25% of 256)                              */
    int32_t decode_quota_max_wg; /* Q_max; 0 = n_workgroups / 2                          */
    int32_t x_moe_expected;   /* x*_moe; <= 0 selects the fixed quota (ratio 1)         */
    int32_t round_multiple;   /* c; 0 = 8 (one workgroup per XCD)                       */
    int32_t group_row_tiles;  /* most row tiles of one expert whose tiles run column
                                 block by column block together, so one fetch of a
                                 weight slice serves all of them; 0 = 8, max 64     */
    const uint32_t* abort_word;   /* NULL, or host/peer-writable: non-zero stops the
                                     kernel at the next tile boundary (MOE_ERR_ABORTED) */
    moe_trace_rec* trace;     /* NULL, or [trace_capacity] records, split into one block
                                 of trace_capacity / W records per workgroup (W = the
                                 launch's workgroups): workgroup w writes its tiles in
                                 order into block w and, if the block has room left,
                                 ends them with a record whose op is -1; tiles past a
                                 full block are not recorded.  trace_capacity >= W.  */
    int64_t trace_capacity;
    moe_op_stats* op_stats;   /* NULL, or [n_ops]                                       */
    int64_t spin_limit;       /* bounded waits, in polls; 0 = default (about 2 s)       */
    int32_t static_partition; /* 0: tile-level sharing as above.  1: a static split for
                                 comparison (the analogue of fixed SM partitions such
                                 as Green Contexts): workgroups below the fixed q' take
                                 only decode tiles, the others only prefill tiles, and
                                 neither borrows idle workgroups of the other phase   */
    int32_t prefill_tile_rows;/* 0 or 192: bf16 prefill ops run 192-row tiles (Eq. (3)'s
                                 M_t = 192).  128: they run the 128-row tiles, which
                                 shortens the longest prefill tile a decode op can wait
                                 for ("Bounded Tile-level Preemption") at some cost in
                                 prefill throughput                                   */
} moe_sched_config;

/* Segment alignment the FFN needs for ops of this phase and dtype (32 rows,
 * one MFMA row block); moe_permute's row_align for such an op must equal it.
 * The FFN cuts an expert's m rows into ceil(m / M_t) row tiles of near-equal
 * height in whole 32-row blocks, M_t = moe_ffn_tile_shape's bm.  Returns
 * <= 0 if unsupported. */
int32_t moe_ffn_row_align(moe_phase_t phase, moe_dtype_t dtype);

/* Output tile of the FFN kernel for ops of this phase and dtype: at most *bm
 * rows (Eq. 3's M_t), *bn columns (GEMM-1: bn/2 gate + bn/2 up columns,
 * i.e. bn/2 columns of h; GEMM-2: bn columns of y_perm), *bk the K step.
 * An op with footprint x_moe (Eq. 3) runs x_moe*(I/(bn/2)) GEMM-1 tiles and
 * x_moe*(H/bn) GEMM-2 tiles.  Returns MOE_OK or MOE_ERR_UNSUPPORTED. */
moe_status_t moe_ffn_tile_shape(moe_phase_t phase, moe_dtype_t dtype, int32_t* bm, int32_t* bn, int32_t* bk);

/* Device scratch needed by one persistent launch over these ops (host array). */
size_t moe_ffn_workspace_bytes(const moe_op_desc* ops, int32_t n_ops, const moe_sched_config* cfg);

/* Launch the adaptive persistent kernel over n_ops operations (ops, cfg: host
 * pointers, read before the call returns).  status_word is a device i32 that
 * this call resets to MOE_OK (on the stream) and the kernel sets to the first
 * data-dependent error.  workspace is moe_ffn_workspace_bytes() bytes. */
moe_status_t moe_grouped_ffn_persistent(const moe_op_desc* ops, int32_t n_ops,
                                        const moe_sched_config* cfg, void* workspace,
                                        int32_t* status_word, void* stream);

/* Comparison baseline (Evaluation, "Overhead of Tile-Level Scheduling": the
 * persistent kernel against plain grouped-GEMM launches): the same tiles as
 * moe_grouped_ffn_persistent with no device scheduler.  Per op, in op order:
 * one planning kernel (the row-tile table of Eq. (3)), one GEMM-1 grid and one
 * GEMM-2 grid (the kernel boundary is the dependency between them), each grid
 * one workgroup per CU taking tiles round robin, column block major.  Readiness
 * fields, the decode quota and the fused combine (moe_op_desc.y) are ignored;
 * h and y_perm equal the persistent kernel's bit for bit.  workspace:
 * moe_ffn_workspace_bytes() bytes; status_word is reset by the first launch. */
moe_status_t moe_grouped_ffn_plain(const moe_op_desc* ops, int32_t n_ops, void* workspace, int32_t* status_word,
                                   void* stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation: the same
 * launch as moe_grouped_ffn_persistent (same kernels, results, readiness and
 * error reporting), with the scheduler workspace in a static device array of
 * the library (MOE_FFN_NOALLOC_WORKSPACE_BYTES per GPU, held until the
 * process ends) instead of a caller-allocated one.  The caller still passes
 * every input and output buffer.  Returns MOE_ERR_CAPACITY before anything is
 * launched when moe_ffn_workspace_bytes(ops) exceeds the array (about 16
 * operations of 250000 rows of capacity each).  Every call on one GPU uses
 * that GPU's array, which keeps the last call's contents and is re-zeroed by
 * each launch: calls that overlap in time on one GPU (different streams, or
 * different threads) race and must not be issued. */
#define MOE_FFN_NOALLOC_WORKSPACE_BYTES (4u << 20)
moe_status_t moe_grouped_ffn_persistent_noalloc(const moe_op_desc* ops, int32_t n_ops,
                                                const moe_sched_config* cfg, int32_t* status_word, void* stream);

/* Weight layout streamed by the FFN kernel (one-time conversion, outside the
 * hot path).  A matrix [N, K] is cut into 32-row blocks of 4 KB chunks, each
 * chunk holding exactly the 16-byte pieces lanes 0..63 feed to the MFMAs of
 * that chunk, so each 64-lane load reads 1 KB contiguous:
 *  bf16: chunk c (64 elements of K) of block b holds, for q = 0..3 and
 *        lane = 0..63 in that order, row 32*b + lane%32, elements
 *        64*c + (lane/32)*32 + 8*q .. +8 (one 32x32x16 MFMA per q);
 *  fp8 e4m3: chunk c (128 elements of K, one scale block) holds, for
 *        kk = 0..1, half = 0..1 and lane = 0..63 in that order, row
 *        32*b + lane%32, elements 128*c + 64*kk + (lane/32)*32 + 16*half .. +16
 *        (one 32x32x64 MFMA per kk).
 * The packed matrix has the same size as the row-major one and block b starts
 * at the same byte offset as row 32*b.  Scales (fp8) are not moved.
 *  src  [E, N, K] row-major (device);  dst  same size (device, not aliasing src)
 * Limits: dtype MOE_BF16 (K % 64 == 0) or MOE_FP8_E4M3 (K % 128 == 0); N % 32 == 0. */
moe_status_t moe_pack_weights(const void* src, void* dst, int32_t E, int32_t N, int32_t K, moe_dtype_t dtype,
                              void* stream);

/* ------------------------------------------------------------------------- a7
 * Weighted combine (Background, "MoE LLM Inference": the chosen experts'
 * outputs are combined before the next layer):
 *   y[t] = sum over j ascending with assign_to_row[t*top_k+j] >= 0 of
 *          topk_w[t*top_k+j] * y_perm[assign_to_row[t*top_k+j]]
 * accumulated in fp32.  A token with no local slot gets exactly 0.
 *  y_perm [*, H] bf16; assign_to_row [T*top_k]; topk_w [T*top_k] f32
 *  y      [T, H] out, y_dtype MOE_BF16 (round to nearest even) or MOE_F32
 * Limits: H a multiple of 8, 1 <= top_k <= 32.
 */
moe_status_t moe_combine(const void* y_perm, const int32_t* assign_to_row, const float* topk_w,
                         int32_t T, int32_t top_k, int32_t H, void* y, moe_dtype_t y_dtype,
                         void* stream);

/* The same combine for up to MOE_MAX_OPS operations in ONE launch: each entry
 * is one moe_combine call's arguments, same meaning, limits and results
 * (bitwise); all entries take the same y_dtype.  ops: host array of n_ops
 * entries, read before the call returns; argument errors of any entry are
 * returned before anything is launched. */
typedef struct moe_combine_args {
    const void* y_perm;
    const int32_t* assign_to_row;
    const float* topk_w;
    int32_t T, top_k, H;
    moe_dtype_t y_dtype;
    void* y;
} moe_combine_args;
moe_status_t moe_combine_batch(const moe_combine_args* ops, int32_t n_ops, void* stream);

/* ------------------------------------------------------------------------- host helpers
 * Pure host arithmetic shared with the kernels (no device access):
 * Eq. (3) footprint over host counts, and Eq. (4) quota in workgroups. */
int32_t moe_x_moe(const int32_t* counts_host, int32_t E_local, int32_t M_t);
int32_t moe_decode_quota(int32_t q, int32_t x_moe, int32_t x_moe_expected, int32_t q_max,
                         int32_t round_multiple);

/* The tile layout the persistent kernel builds when it instantiates one
 * operation ("Tile-Level Scheduling"; Eq. (3)), computed on the host with the
 * kernel's own index arithmetic, for inspection and testing:
 *  counts, offsets  [E_local], [E_local] host arrays (as moe_permute writes them)
 *  M_t              the op class's row-tile height (moe_ffn_tile_shape bm)
 *  gmax             group_row_tiles (the kernel's default is 8)
 *  n1, n2           GEMM-1 / GEMM-2 column blocks (I/(bn/2), H/bn)
 * Writes, for each row tile p < x_moe: row_tiles[4p..4p+3] = expert, row tile
 * within the expert, valid rows, first row; groups[2p..2p+1] = first row
 * tile and size of its weight-sharing group; for each XCD queue x < 8:
 * queues[2x..2x+1] = first row tile, row tiles; and for every tile of every
 * queue in claim order: tiles[4i..4i+3] = queue, stage (1 or 2), row tile,
 * column block.  Returns x_moe, -1 on bad arguments or too small arrays
 * (max_row_tiles entries of row_tiles/groups, max_tiles of tiles), -2 if a
 * claim would resolve differently on workgroups of different XCDs. */
int32_t moe_sched_layout(const int32_t* counts, const int32_t* offsets, int32_t E_local, int32_t M_t, int32_t gmax,
                         int32_t n1, int32_t n2, int32_t max_row_tiles, int32_t* row_tiles, int32_t* groups,
                         int32_t* queues, int64_t max_tiles, int32_t* tiles);

/* sizeof() of the ABI structs, so bindings can check their layout:
 * 0 moe_op_desc, 1 moe_sched_config, 2 moe_trace_rec, 3 moe_op_stats,
 * 4 moe_route_args, 5 moe_permute_args, 6 moe_combine_args; 0 otherwise. */
size_t moe_abi_sizeof(int32_t which);

const char* moe_status_string(moe_status_t status);
const char* moe_last_error(void);   /* thread-local message of the last failing call */

#ifdef __cplusplus
}
#endif
#endif /* MOE_APK_H */
