/*
 * moe_stage.h - C ABI of the MI355X (gfx950) MoE expert stage.
 *
 * The stage is the data-parallel work one device runs on its own share of the
 * experts of a MoE layer in a disaggregated attention/MoE prefill system
 * (paper: "ASAP: A Disaggregated and Asynchronous Inference System for MoE
 * Prefill", sections 3.2 and 3.4).  Token micro-batches arrive with top-k
 * expert ids; the stage
 *   1. groups their slots by local expert with a stable counting sort
 *      (the per-expert token counts are the dispatch metadata of section
 *      3.2.1 and Table 2),
 *   2. runs each local expert's SwiGLU FFN as a grouped matrix
 *      multiplication, hidden states on the left and the expert's weights on
 *      the right (section 3.4.2, "Bubble-Free Kernel Dispatching"),
 *   3. reduces the k expert results of each token with its routing weights
 *      back into token order (section 3.2.2; Table 2 stores k result rows per
 *      token), and
 *   4. does all of it on the caller's stream per micro-batch, without any
 *      device-wide barrier or host read-back (sections 3.4.1 and 3.4.2).
 * A stage may hold the expert weights of several layers (the MoE Super
 * Kernel of section 3.4.2: weights of all L layers resident, an on-device
 * table of their addresses, the layer id a device-side argument): a
 * micro-batch then names its layer through a device pointer that the GEMM
 * kernels read when they run, so work for any layer can be enqueued ahead
 * of time without the host knowing which layer it is.
 *
 * Conventions (section 3.2: buffers are allocated once at initialisation and
 * live as long as the framework; weights stay resident in HBM):
 *   - moe_stage_create copies the weights into stage-owned device memory and
 *     allocates every workspace buffer; no enqueue call allocates memory.
 *   - All pointers in moe_weights / moe_microbatch are DEVICE pointers.
 *     Micro-batch buffers are borrowed: they must stay valid and unmodified
 *     until the work enqueued on `stream` has completed.
 *   - `stream` is a hipStream_t passed as void*; NULL means the default stream.
 *   - Enqueue calls are asynchronous.  Host-detectable errors are returned
 *     synchronously and then NOTHING has been enqueued.  Expert ids outside
 *     [-1, n_experts) are detected on the device: the slot is skipped (as if
 *     masked) and a sticky error word is set that moe_stage_sync reports.
 *   - Layouts are row-major.  bf16 is the IEEE-754 binary32 upper half;
 *     fp8 is OCP E4M3FN (bias 7, max 448, no infinities).
 *
 * Definition of the outputs, for one micro-batch of T tokens with ids[T][k]
 * (slot s = t*k + j) and local experts [e0, e0 + E_loc):
 *   counts[e]      number of slots with id e, e in [0, n_experts)
 *   offsets[i]     sum_{i' < i} counts[e0 + i'], i in [0, E_loc]
 *   slot_of_row[r] local slots in ascending (expert id, s) order
 *   row_of_slot[s] row of slot s in that order, -1 if s is not local
 *   y_r            = W_down (SiLU(W_gate x_t) * (W_up x_t)), t = slot_of_row[r] / k
 *   out[t]         = base_t + sum_{j ascending, row_of_slot[t*k+j] >= 0}
 *                            w[t][j] * y_{row_of_slot[t*k+j]}
 *   base_t         = 0 (MOE_COMBINE_OVERWRITE) or the previous out[t]
 *                    (MOE_COMBINE_ACCUMULATE), plus the shared expert's
 *                    output when the stage has one.
 * Intermediate rows (H, Y_perm) are stored in bf16 (fp8 mode: H as e4m3
 * with per-128-channel fp32 scales; h is quantised from its fp32 value by
 * the rule of moe_quantize_fp8).  X_perm is never materialised: the gate/up
 * grouped GEMM loads row r straight from x[slot_of_row[r] / k] (the row
 * gather is fused into its token-row loads); in fp8 mode only the rows'
 * scales are gathered, transposed, into x_perm_scales.  The combine accumulates in
 * fp32 and rounds once to bf16.  Tokens with no local slot are written as
 * +0.0 (overwrite) or left untouched (accumulate).  The combine uses no
 * atomics, so results are bit-identical from run to run and independent of
 * how micro-batches are spread over streams.
 */
#ifndef MOE_STAGE_H
#define MOE_STAGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_API __attribute__((visibility("default")))

/* Opaque stage handle, owned by the library (create / destroy). */
typedef struct moe_stage moe_stage;

typedef int32_t moe_status;
#define MOE_OK              0
#define MOE_EINVAL         (-1)   /* bad argument (null pointer, bad slot, size) */
#define MOE_ENOMEM         (-2)   /* device allocation failed in create */
#define MOE_EHIP           (-3)   /* a HIP runtime call failed */
#define MOE_EBADID         (-4)   /* device saw an expert id outside [-1, n_experts) */
#define MOE_EUNSUPPORTED   (-5)   /* shape or mode the library does not support */
#define MOE_EBUSY          (-6)   /* slot still in flight (moe_stage_poll) */
#define MOE_EBADLAYER      (-7)   /* device saw a layer id outside [0, n_layers) */
#define MOE_ETIMEOUT       (-8)   /* an ingest wait gave up (moe_ingest_wait) */
#define MOE_EBADCOUNT      (-9)   /* device saw pre-grouped counts that are negative or
                                     overrun the rows buffer (moe_expert_ffn_grouped) */

enum { MOE_DTYPE_BF16 = 0, MOE_DTYPE_FP8_E4M3_B128 = 1 };
enum { MOE_COMBINE_OVERWRITE = 0, MOE_COMBINE_ACCUMULATE = 1 };

/* Stage shape.  Requirements: d_model and d_ff multiples of 128;
 * 1 <= n_experts <= 1024; 0 <= first_local_expert;
 * 1 <= n_local_experts <= 256; first_local_expert + n_local_experts <=
 * n_experts; 1 <= top_k <= 32; 0 <= max_tokens with max_tokens * d_model * 2
 * < 2^31 (token rows are addressed with 32-bit offsets); 1 <= n_slots <= 64;
 * 1 <= n_layers <= 1024 (every layer has the same shape and local experts). */
typedef struct {
    int32_t d_model;             /* hidden size d (paper: H) */
    int32_t d_ff;                /* expert intermediate size f */
    int32_t n_experts;           /* routed experts in the model (paper: E_total) */
    int32_t first_local_expert;  /* e0 */
    int32_t n_local_experts;     /* E_loc */
    int32_t top_k;               /* k */
    int32_t max_tokens;          /* largest micro-batch (paper: S) */
    int32_t n_slots;             /* micro-batches that may be in flight at once */
    int32_t dtype;               /* MOE_DTYPE_* */
    int32_t has_shared_expert;   /* 1: one always-on shared SwiGLU expert */
    int32_t n_layers;            /* layers whose weights the stage holds (paper: L) */
} moe_stage_desc;

/* Expert weights of one layer (device pointers; read during create only;
 * moe_stage_create takes an array of n_layers of them, layer 0 first).
 * bf16:  w_gate, w_up [E_loc][f][d] bf16; w_down [E_loc][d][f] bf16.
 * fp8:   the same shapes as e4m3 bytes, with fp32 scales per 128x128 block:
 *        s_gate, s_up [E_loc][f/128][d/128], s_down [E_loc][d/128][f/128].
 * sh_*:  the shared expert, same layout with E_loc = 1 (NULL if none). */
typedef struct {
    const void  *w_gate, *w_up, *w_down;
    const float *s_gate, *s_up, *s_down;
    const void  *sh_gate, *sh_up, *sh_down;
    const float *sh_s_gate, *sh_s_up, *sh_s_down;
} moe_weights;

/* One micro-batch (device pointers).
 * x:        [T][d] bf16, or [T][d] e4m3 in fp8 mode
 * x_scales: fp8 mode only, [T][d/128] fp32 (see moe_quantize_fp8)
 * topk_ids: [T][k] int32, -1 = masked slot
 * topk_w:   [T][k] fp32 routing weights
 * out:      [T][d] bf16
 * layer_id: one int32 in device memory, the layer whose weights the GEMMs
 *           use, read on the device when they run (so it may be written by
 *           earlier work on the stream after the host enqueued this
 *           micro-batch); NULL means layer 0.  A value outside
 *           [0, n_layers) is clamped into range and reported by
 *           moe_stage_sync as MOE_EBADLAYER. */
typedef struct {
    int32_t        n_tokens;
    const void    *x;
    const float   *x_scales;
    const int32_t *topk_ids;
    const float   *topk_w;
    void          *out;
    int32_t        combine_mode;   /* MOE_COMBINE_* */
    const int32_t *layer_id;
} moe_microbatch;

/* A batch of rows that arrives already grouped by local expert: the receive
 * region of section 3.2.1 in the form Table 2 gives it on the MoE side, with
 * the senders' per-expert token counts as metadata and one payload row per
 * (token, local expert) pair.  Device pointers.
 * rows:       [n_rows_max][d] bf16, or e4m3 in fp8 mode; the rows of local
 *             expert i are rows [c_0 + ... + c_{i-1}, + c_i), c = counts
 * row_scales: fp8 mode only, [n_rows_max][d/128] fp32 (moe_quantize_fp8)
 * counts:     [n_local_experts] int32, read on the device when the work runs
 *             (the host never learns them); a negative count is taken as 0
 *             and rows past n_rows_max are dropped (trailing experts lose
 *             rows), both reported by moe_stage_sync as MOE_EBADCOUNT
 * y:          [n_rows_max][d] bf16: y_r = W_down (SiLU(W_gate x_r) * (W_up x_r))
 *             with the weights of the row's expert; rows past the counted
 *             total are not written.  The routing weights are not applied:
 *             the weighted sum over a token's k results is formed where the
 *             results return to (section 3.2.2).
 * n_rows_max: rows the buffers hold, 0 <= n_rows_max <= capacity_rows
 * layer_id:   as in moe_microbatch (NULL: layer 0) */
typedef struct {
    int32_t        n_rows_max;
    const void    *rows;
    const float   *row_scales;
    const int32_t *counts;
    void          *y;
    const int32_t *layer_id;
} moe_grouped_batch;

/* Device pointers into one slot's workspace (for tests and inspection).
 * Valid after the slot's work has completed; overwritten by its next use. */
typedef struct {
    int32_t *counts;          /* [n_experts] */
    int32_t *offsets;         /* [E_loc + 1] */
    int32_t *slot_of_row;     /* [capacity_rows] */
    int32_t *row_of_slot;     /* [max_tokens * k] */
    void    *x_perm;          /* NULL: the row gather is fused into the gate/up GEMM */
    float   *x_perm_scales;   /* fp8: the routed rows' x scales, [d/128][capacity_rows] (transposed) */
    void    *h;               /* [capacity_rows][f] bf16 or e4m3 */
    float   *h_scales;        /* fp8: [f/128][capacity_rows] (transposed) */
    void    *y_perm;          /* [capacity_rows][d] bf16 */
    void    *h_shared;        /* shared expert: [max_tokens][f] */
    float   *h_shared_scales; /* fp8 shared expert: [f/128][max_tokens] (transposed) */
    void    *y_shared;        /* shared expert: [max_tokens][d] bf16 */
    int32_t  capacity_rows;   /* max_tokens * k */
    int32_t  n_tokens;        /* T of the micro-batch last dispatched here */
} moe_dispatch_view;

/* Validates `desc` (MOE_EUNSUPPORTED when d_model or d_ff is not a multiple
 * of 128, MOE_EINVAL for any other bad field), copies the weights of its
 * n_layers layers
 * (weights[0 .. n_layers-1]) into stage-owned HBM, packed for the grouped
 * GEMM, builds the on-device table of the layers' weight addresses, and
 * allocates all workspace for n_slots micro-batches of up to max_tokens
 * tokens.  Synchronous.  On error *out is NULL. */
MOE_API moe_status moe_stage_create(const moe_stage_desc *desc, const moe_weights *weights,
                            moe_stage **out);

/* Waits for all work of the stage and frees it.  NULL is a no-op. */
MOE_API void moe_stage_destroy(moe_stage *stage);

/* Step 1 (histogram, scan, stable scatter; in fp8 mode also the gather of
 * the routed rows' scales into x_perm_scales) on `slot`'s workspace.  Records
 * the micro-batch for the slot's later calls: the gate/up GEMM of
 * moe_expert_ffn reads the token rows from mb->x, which must stay valid until
 * the slot's work completes (as every micro-batch buffer must). */
MOE_API moe_status moe_dispatch(moe_stage *stage, int32_t slot, const moe_microbatch *mb,
                        void *stream);

/* Step 2: grouped GEMM gate/up with fused SiLU*up epilogue, then grouped GEMM
 * down, for every local expert with rows (and the shared expert, if any).
 * The tile schedule is built on the device by moe_dispatch. */
MOE_API moe_status moe_expert_ffn(moe_stage *stage, int32_t slot, void *stream);

/* Step 2 for pre-grouped rows (moe_grouped_batch): builds the tile tables
 * on the device from gb->counts, then runs the same grouped GEMMs as
 * moe_expert_ffn on gb->rows into gb->y, on `slot`'s workspace (H; fp8 also
 * the transposed row scales).  The stage's shared expert, if any, is not
 * run (it applies to tokens, not to routed rows).  The slot then holds no
 * micro-batch: moe_combine on it returns MOE_EINVAL until the next
 * moe_dispatch.  Host errors (null pointers with n_rows_max > 0, a bad slot,
 * n_rows_max outside [0, capacity_rows]) return MOE_EINVAL, enqueueing
 * nothing. */
MOE_API moe_status moe_expert_ffn_grouped(moe_stage *stage, int32_t slot,
                                          const moe_grouped_batch *gb, void *stream);

/* Step 3: weighted combine into mb->out (deterministic, no atomics). */
MOE_API moe_status moe_combine(moe_stage *stage, int32_t slot, void *stream);

/* Steps 1-3 on `stream` for one micro-batch, on the next slot of the
 * stage's ring.  Never blocks the host: if that slot's previous micro-batch
 * may still be in flight, `stream` first waits on the device for exactly that
 * one (the backpressure of section 3.2.1, without a global barrier).
 * *slot_out (may be NULL) receives the slot used. */
MOE_API moe_status moe_stage_submit_microbatch(moe_stage *stage, const moe_microbatch *mb,
                                       void *stream, int32_t *slot_out);

/* Sender-side activation quantiser for the fp8 variant: per token, per 128
 * channels, scale = amax / 448 in fp32 (1 if amax = 0), code = e4m3 of
 * x / scale (fp32 division, round to nearest even).  x_bf16 [T][d],
 * x_q [T][d] bytes, x_s [T][d/128] fp32.  d must be a multiple of 128. */
MOE_API moe_status moe_quantize_fp8(const void *x_bf16, int32_t n_tokens, int32_t d_model,
                            void *x_q, float *x_s, void *stream);

/* Asynchronous ingest (section 3.2.1; the per-sender ready bits of Table 2).
 * The senders of a micro-batch write their token rows, ids and weights into
 * receive buffers that live as long as the stage (the moe_microbatch
 * pointers), then each raises its ready word with moe_ingest_signal.
 * moe_ingest_wait enqueues on `stream` a wait, on the device, until every
 * ready[i], i < n_words, has reached `epoch` (compared as a wrapping 32-bit
 * round counter, so the words never need clearing); work enqueued on
 * `stream` after it -- typically moe_stage_submit_microbatch, enqueued long
 * before the rows arrive -- starts as soon as they have, with no host round
 * trip.  The wait runs as one wave polling the words and is bounded: after
 * spin_limit polls (0: about one second) it gives up, the work after it runs
 * on whatever the buffers hold, and the next moe_stage_sync (once that work
 * has been waited for) returns MOE_ETIMEOUT.  ready: device memory,
 * 1 <= n_words <= 4096. */
MOE_API moe_status moe_ingest_wait(moe_stage *stage, const uint32_t *ready, int32_t n_words,
                           uint32_t epoch, uint32_t spin_limit, void *stream);

/* Enqueues on `stream`, after its earlier work, a store of `epoch` into the
 * device word *word with release order: a sender raising its ready word once
 * its rows are written, or the MoE side acknowledging a consumed round so the
 * senders may overwrite the buffers (backpressure). */
MOE_API moe_status moe_ingest_signal(uint32_t *word, uint32_t epoch, void *stream);

/* Non-blocking test of one slot (section 3.2.1: a receiver looks at a
 * region without waiting for it): MOE_OK when the work last enqueued on
 * `slot` has completed (or the slot was never used), MOE_EBUSY while it is
 * still in flight, MOE_EINVAL for a bad slot.  Never waits and never
 * enqueues anything; the host may use it to pick a free slot or to decide
 * whether the next submit would make its stream wait. */
MOE_API moe_status moe_stage_poll(moe_stage *stage, int32_t slot);

/* The dispatch index of moe_dispatch (histogram over all experts, offsets,
 * stable counting-sort permutation; bf16 moe_dispatch minus the stage) for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  Allocates nothing:
 * its only scratch (one histogram row of n_experts counts per 1024 slots,
 * and the grouped-GEMM tile tables) is a fixed 4 MiB array that the library
 * holds on every device it runs on until the process ends.
 * Inputs:  topk_ids [n_tokens][top_k] int32 (-1 = masked), device memory.
 * Outputs (device memory, written as moe_dispatch writes them into a slot):
 *   counts [n_experts], offsets [n_local_experts + 1],
 *   slot_of_row [n_tokens * top_k] (the first offsets[n_local_experts]
 *   entries are written), row_of_slot [n_tokens * top_k].
 * err: optional device int32; an expert id outside [-1, n_experts) sets
 *   bit 0 (the slot is skipped); the caller clears it.  NULL: not reported.
 * Errors: MOE_EINVAL for bad sizes or null pointers; MOE_EUNSUPPORTED when
 * ceil(n_tokens * top_k / 1024) * n_experts > 2^20 (the scratch holds no
 * more histogram rows); nothing is enqueued then.  Every call on a device
 * shares that device's scratch array: calls that overlap on one device
 * (two streams, two threads) race and must be serialised by the caller.
 * `stream` must belong to the current device. */
MOE_API moe_status moe_dispatch_index_noalloc(const int32_t *topk_ids, int32_t n_tokens,
                                              int32_t top_k, int32_t n_experts,
                                              int32_t first_local_expert, int32_t n_local_experts,
                                              int32_t *counts, int32_t *offsets,
                                              int32_t *slot_of_row, int32_t *row_of_slot,
                                              int32_t *err, void *stream);

/* A stream whose kernels may run only on the current device's compute units
 * [first_cu, first_cu + n_cus) (mask bits in the runtime's CU order), so
 * dispatch and combine can be given their own share of the CUs beside the
 * grouped GEMMs (section 3.4.1: compute and communication streams each own
 * a partition of the cores).  The stage's persistent kernels size their
 * grids by the CUs of the stream they are launched on.  Each such stream
 * takes a hardware queue of its own: with the runtime's default of four
 * queues per process, create at most three, before any other stream.
 * MOE_EINVAL for a null out or a range outside the device; MOE_ENOMEM when
 * no hardware queue is left.  Destroy with moe_stream_destroy, which waits
 * for the stream's work first. */
MOE_API moe_status moe_stream_create_cu_masked(int32_t first_cu, int32_t n_cus, void **stream_out);
MOE_API moe_status moe_stream_destroy(void *stream);

/* Fills `out` with the device pointers of `slot`'s workspace. */
MOE_API moe_status moe_stage_query(moe_stage *stage, int32_t slot, moe_dispatch_view *out);

/* Waits until every slot's enqueued work has completed and returns (then
 * clears) the sticky device errors: MOE_EBADID if a kernel saw an invalid
 * expert id since the last sync, else MOE_EBADLAYER if one saw an invalid
 * layer id, else MOE_EBADCOUNT if one saw invalid pre-grouped counts, else
 * MOE_ETIMEOUT if an ingest wait gave up, else MOE_OK (or MOE_EHIP). */
MOE_API moe_status moe_stage_sync(moe_stage *stage);

/* Per-kernel timing with HIP events, for measurement (off by default).
 * While enabled, every enqueue call records an event pair around each of its
 * kernel groups on the launch stream (this creates events, i.e. allocates
 * host-side runtime objects).  Kinds, in order: 0 dispatch index
 * (histogram, scan, scatter), 1 gather of the token scales (fp8 only; the
 * rows themselves are gathered inside kind 2), 2 grouped GEMM gate/up with the SiLU*up epilogue (fp8: and the
 * quantisation of h), 3 grouped GEMM down, 4 combine, 5 reserved (no
 * longer recorded). */
#define MOE_PROF_KINDS 6
MOE_API moe_status moe_stage_profile(moe_stage *stage, int32_t enable);

/* Waits for the recorded events, writes the summed milliseconds and the
 * number of timed launches per kind into ms[MOE_PROF_KINDS] and
 * launches[MOE_PROF_KINDS], and clears the records. */
MOE_API moe_status moe_stage_profile_read(moe_stage *stage, double *ms, int32_t *launches);

/* Bytes of device memory moe_stage_create allocates for `desc` (weights plus
 * workspace).  Host-only arithmetic; needs no GPU. */
MOE_API moe_status moe_stage_workspace_bytes(const moe_stage_desc *desc, int64_t *bytes);

/* Static text for a status code. */
MOE_API const char *moe_status_string(moe_status status);

#ifdef __cplusplus
}
#endif

#endif /* MOE_STAGE_H */
