/*
 * turbosparse.h — C ABI of the MI355X (gfx950) activation-sparse dReLU
 * feed-forward library.
 *
 * The operation (Turbo Sparse, arXiv 2406.05955):
 *   Eq. (gated-MLP), section 2, with F_act = ReLU applied to BOTH projections
 *   (Eq. (drelu), section 3.2; no bias, section 3.2 footnote):
 *       Combined(x) = max(0, x W_gate) * max(0, x W_up)
 *       out(x)      = Combined(x) W_down
 *   A neuron whose Combined activation is zero contributes nothing (sections
 *   1 and 6.2), so the sparse entry points read a W_up row only for neurons
 *   whose gate is positive, and a W_down row only for neurons whose Combined
 *   activation is non-zero.  The result equals the dense definition exactly
 *   up to floating-point summation order.
 *   MoE form (section 6.2, "2 out of 8 experts"): a router picks top_k experts
 *   per token and each routed expert is a dReLU FFN.  Router details, which
 *   the paper leaves to Mixtral: logits = W_r x, p = softmax(logits), the
 *   top_k largest p (lower expert index wins exact ties), weights
 *   w = p / sum(p over the chosen experts), out = sum_k w_k FFN_{e_k}(x).
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller.  The
 *     library allocates and frees nothing; scratch memory is the caller's
 *     workspace `ws` of `ws_bytes` bytes (query the size first).
 *   - Layout: x and out are fp32 row-major [batch][hidden].  Every weight
 *     matrix is neuron-major [inter][hidden], row-major, in `wdtype`
 *     (TS_F32: float, TS_BF16: bfloat16 bit patterns, 2 bytes).  Row i of
 *     w_down_t is neuron i's output row, i.e. the paper's W_down row i.
 *     MoE experts are packed [n_experts][inter][hidden]; the router is
 *     [n_experts][hidden] in `wdtype`.
 *   - Arithmetic: fp32 accumulation; x, the gate / up projections and
 *     Combined stay fp32.  An active set is defined by strict comparisons
 *     (gate > 0; Combined non-zero iff gate > 0 and up > 0).
 *   - `out` is overwritten, never accumulated into.
 *   - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *     NULL = the default stream); results are valid after the caller
 *     synchronises that stream.  Concurrent calls need distinct workspaces.
 *     Workspace contents after a call are unspecified.
 *   - All argument checks run on the host before anything is enqueued.  On
 *     any error the call returns a non-zero ts_status, enqueues nothing and
 *     leaves every output untouched.  A failed kernel launch returns
 *     TS_ERR_HIP (ts_last_error() has the HIP message).  Errors during
 *     execution surface at the caller's stream synchronisation.
 *   - Constraints: 1 <= batch <= 256; inter >= 1; hidden >= 8 and
 *     hidden % 8 == 0 (TS_BF16) or hidden % 4 == 0 (TS_F32); hidden <= 8192
 *     (TS_BF16) or <= 4096 (TS_F32); 1 <= n_experts <= 64;
 *     1 <= top_k <= min(n_experts, 8); x, weights, out and ws 16-byte
 *     aligned; topk_idx, topk_w and the stats arrays 4-byte aligned.
 *   - Non-finite inputs give unspecified (but memory-safe) results.
 *   - No exceptions cross this interface.
 */
#ifndef TURBOSPARSE_H
#define TURBOSPARSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TS_OK = 0,
    TS_ERR_NULL = 1,        /* a required pointer is NULL */
    TS_ERR_SHAPE = 2,       /* batch / hidden / inter / n_experts / top_k out of range */
    TS_ERR_DTYPE = 3,       /* unknown ts_dtype */
    TS_ERR_ALIGN = 4,       /* a pointer is not 16-byte aligned */
    TS_ERR_WORKSPACE = 5,   /* ws is NULL or ws_bytes is below the required size */
    TS_ERR_HIP = 6,         /* a HIP runtime call or kernel launch failed */
    TS_ERR_UNSUPPORTED = 7  /* valid request the library does not serve (e.g. stats on a dense call) */
} ts_status;

typedef enum { TS_F32 = 0, TS_BF16 = 1 } ts_dtype;

/*
 * Optional per-token activity report (device pointers, each nullable).  For
 * ts_ffn_sparse, "token" t indexes the batch; for ts_moe_sparse the report is
 * per (token, routed slot) pair, index t * top_k + k, slot k in rank order.
 *   n_gate[t]      |G_t|, G_t = {i : gate_{t,i} > 0}
 *   n_active[t]    |A_t|, A_t = {i : gate_{t,i} > 0 and up_{t,i} > 0}
 *   gate_idx[t*inter .. t*inter + n_gate[t])      G_t ascending
 *   active_idx[t*inter .. t*inter + n_active[t])  A_t ascending
 *   n_union[0..1]  |union_t G_t|, |union_t A_t| over the batch (ts_ffn_sparse
 *                  only; these are the rows the batched path reads)
 * Entries past a token's count are unspecified.  Producing the report costs
 * extra small kernels; leave the pointer NULL on timed paths.
 */
typedef struct {
    int32_t *n_gate;
    int32_t *n_active;
    int32_t *gate_idx;
    int32_t *active_idx;
    int32_t *n_union;
} ts_ffn_stats;

/* Workspace bytes needed by ts_ffn_sparse / ts_ffn_dense for these sizes
 * (0 if the sizes are out of range). */
size_t ts_ffn_workspace_bytes(int batch, int hidden, int inter, ts_dtype wdtype);

/*
 * Activation-sparse dReLU FFN: out[t] = sum_{i in A_t} Combined_{t,i} *
 * w_down_t[i][:], with W_gate read whole and W_up / W_down rows read only for
 * G_t / A_t (Eq. drelu; section 6.2's zero-activation skipping).
 *   x [batch][hidden] fp32; w_gate, w_up, w_down_t [inter][hidden] wdtype;
 *   out [batch][hidden] fp32; stats nullable; ws/ws_bytes workspace;
 *   stream hipStream_t or NULL.
 * batch == 1 uses the pipelined single-token kernel.  batch > 1 with
 * TS_BF16 weights reads every weight row at most once per pass of up to 64
 * tokens (the rows of the union of the pass's active sets) and runs the
 * contraction on the matrix cores, x and Combined entering as high + low
 * bf16 parts (fp32-level accuracy); TS_F32 weights run the single-token
 * kernels per token, and so does a TS_BF16 batch above 64 whose report asks
 * for the union counts (they need a single pass).
 */
ts_status ts_ffn_sparse(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                        ts_dtype wdtype, int batch, int hidden, int inter, float *out,
                        const ts_ffn_stats *stats, void *ws, size_t ws_bytes, void *stream);

/*
 * The dReLU FFN with the top-k magnitude mask (section 3.2, Eq. mask and Eq.
 * sparsify-gated-MLP, the paper's knob for measuring a model at a chosen
 * sparsity): per token only the `keep` largest |Combined| activations enter
 * the down projection (ties: the lower neuron index; keep above the number
 * of non-zero activations keeps them all, i.e. the ts_ffn_sparse result).
 * W_gate is read whole, the W_up rows of G and the W_down_t rows of the
 * kept neurons only.  The activity report's A_t is the kept set (its
 * non-zero members).  keep >= 0 (TS_ERR_SHAPE otherwise); inter <= 16384
 * (TS_ERR_UNSUPPORTED otherwise: the per-token selection runs in on-chip
 * memory).  Other arguments as ts_ffn_sparse, same workspace size.  A call
 * without a report and one with it run different kernel sequences and give
 * the same bits.
 */
ts_status ts_ffn_sparse_topk(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                             ts_dtype wdtype, int batch, int hidden, int inter, int keep, float *out,
                             const ts_ffn_stats *stats, void *ws, size_t ws_bytes, void *stream);

/* Activation of the FFN (ts_ffn_sparse_act). */
typedef enum {
    TS_ACT_DRELU = 0,     /* Eq. drelu: Combined = max(0, gate) * max(0, up) */
    TS_ACT_RELU_GATE = 1  /* gate-only ReLU with threshold tau: Combined = max(0, gate - tau) * up */
} ts_act;

/*
 * The sparse FFN with a choice of activation, to set dReLU beside the
 * ReLUfication baselines of section 3.1: TS_ACT_RELU_GATE with tau = 0 is
 * ReGLU (Eq. gated-MLP with F_act = ReLU, section 2), tau > 0 its shifted
 * form (section 3.1: the threshold of the gate's ReLU moved to mask more of
 * it; read as max(0, gate - tau)).  The up branch is not masked, so a neuron
 * whose gate passes the threshold is active unless its up projection is
 * exactly zero (A = G): W_gate is read whole, and the W_up and W_down_t rows
 * of G.  TS_ACT_DRELU requires tau == 0 and is ts_ffn_sparse.
 * The activity report gives G_t = {gate > tau} and A_t = {Combined != 0}.
 * Other arguments as ts_ffn_sparse, same workspace size.  TS_ACT_RELU_GATE
 * runs the single-token kernels per token (the batched matrix-core path
 * serves dReLU only).  An unknown `act`, a non-finite tau, or a non-zero tau
 * with TS_ACT_DRELU returns TS_ERR_SHAPE.
 */
ts_status ts_ffn_sparse_act(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                            ts_dtype wdtype, int batch, int hidden, int inter, ts_act act, float tau,
                            float *out, const ts_ffn_stats *stats, void *ws, size_t ws_bytes, void *stream);

/*
 * Dense comparator: the same function (Eq. gated-MLP with dReLU) computed
 * over every neuron, reading all three matrices in full.  Same arguments as
 * ts_ffn_sparse without the stats report.
 */
ts_status ts_ffn_dense(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                       ts_dtype wdtype, int batch, int hidden, int inter, float *out, void *ws,
                       size_t ws_bytes, void *stream);

/* Workspace bytes for ts_ffn_sparse_given (0 if out of range). */
size_t ts_ffn_given_workspace_bytes(int batch, int hidden, int inter, int max_count, ts_dtype wdtype);

/*
 * Sparse dReLU FFN over externally supplied neuron lists: the interface an
 * activation predictor drives (section 7 of the paper: the inference engine
 * evaluates only the neurons a predictor marks active, so the gate
 * projection of the other neurons is never read).  For token t only the
 * entries idx[t][0 .. min(count[t], max_count)) are evaluated, in any
 * order: their W_gate and W_up rows are read (together: a listed neuron is
 * predicted active, so the up row is not held back until the gate's sign is
 * known), and the W_down_t rows of those whose Combined activation is
 * non-zero.  Entries outside [0, inter) are skipped; a repeated entry
 * contributes again.  A list that holds every neuron of G_t (for instance
 * the gate_idx report of ts_ffn_sparse) gives the ts_ffn_sparse result up
 * to fp32 summation order; a list that misses active neurons leaves their
 * terms out (the predictor's approximation).
 *   idx   device int32 [batch][max_count]; count device int32 [batch]
 *         (values below 0 count as 0, above max_count as max_count);
 *   stats nullable; only n_gate (listed entries with a positive gate) and
 *         n_active (listed entries with a non-zero Combined activation)
 *         are served, the other stats fields must be NULL
 *         (TS_ERR_UNSUPPORTED otherwise);
 *   other arguments and constraints as ts_ffn_sparse, plus
 *   1 <= max_count <= 2^24, idx and count 4-byte aligned, and rows of at
 *   most 512 16-byte chunks (hidden <= 4096 for TS_BF16, <= 2048 for
 *   TS_F32; TS_ERR_UNSUPPORTED otherwise).
 */
ts_status ts_ffn_sparse_given(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                              ts_dtype wdtype, int batch, int hidden, int inter, const int32_t *idx,
                              const int32_t *count, int max_count, float *out, const ts_ffn_stats *stats,
                              void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes for ts_moe_sparse / ts_moe_dense (0 if out of range). */
size_t ts_moe_workspace_bytes(int batch, int hidden, int inter, int n_experts, int top_k,
                              ts_dtype wdtype);

/*
 * Top-k MoE layer with activation-sparse dReLU experts (section 6.2).
 *   x [batch][hidden] fp32; w_router [n_experts][hidden] wdtype;
 *   w_gate, w_up, w_down_t [n_experts][inter][hidden] wdtype;
 *   out [batch][hidden] fp32;
 *   topk_idx [batch][top_k] int32 (nullable): chosen experts, rank order;
 *   topk_w [batch][top_k] fp32 (nullable): their renormalised weights;
 *   stats (nullable): per (token, slot) report, see ts_ffn_stats;
 *   ws / ws_bytes / stream as above.
 * The routing decision never leaves the device.  Batch 1 (and TS_F32
 * weights) run the pipelined single-token kernel, each workgroup computing
 * its token's router; 2 <= batch <= 64 with TS_BF16 weights run the
 * matrix-core path, each expert's tokens in groups of about twice the
 * expected load (an expert drawing more takes further groups and reads its
 * weights once more per group).
 */
ts_status ts_moe_sparse(const float *x, const void *w_router, const void *w_gate, const void *w_up,
                        const void *w_down_t, ts_dtype wdtype, int batch, int hidden, int inter,
                        int n_experts, int top_k, float *out, int32_t *topk_idx, float *topk_w,
                        const ts_ffn_stats *stats, void *ws, size_t ws_bytes, void *stream);

/*
 * ts_ffn_sparse without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  Arguments, results and errors
 * as ts_ffn_sparse (the same kernels run); the scratch memory is a fixed
 * array of TS_NOALLOC_SCRATCH_BYTES (32 MiB) inside the library, one per
 * GPU, which each GPU the library runs on holds until the process ends.
 * The first call on a device looks up that device's array (no allocation);
 * the device current on the calling thread must be the one holding the
 * pointers and the stream.  Shapes whose workspace (ts_ffn_workspace_bytes)
 * exceeds the array are rejected with TS_ERR_WORKSPACE before anything is
 * enqueued (at hidden 4096, inter 14336, bf16: batch <= 4 fits).
 * Every call on one GPU uses the same array: calls that overlap in time on
 * one GPU (several streams, several host threads) race and give undefined
 * results; serialise them.  No state carries over between calls: each
 * call writes all the scratch it reads.
 */
#define TS_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
ts_status ts_ffn_sparse_noalloc(const float *x, const void *w_gate, const void *w_up, const void *w_down_t,
                                ts_dtype wdtype, int batch, int hidden, int inter, float *out,
                                const ts_ffn_stats *stats, void *stream);

/* Dense comparator of ts_moe_sparse: same routing, every routed expert
 * computed densely.  Same arguments without the stats report. */
ts_status ts_moe_dense(const float *x, const void *w_router, const void *w_gate, const void *w_up,
                       const void *w_down_t, ts_dtype wdtype, int batch, int hidden, int inter,
                       int n_experts, int top_k, float *out, int32_t *topk_idx, float *topk_w,
                       void *ws, size_t ws_bytes, void *stream);

/* Human-readable name of a status code (static string). */
const char *ts_status_str(ts_status s);

/* Message of the last TS_ERR_HIP on the calling thread ("" if none). */
const char *ts_last_error(void);

/* Library version string (static). */
const char *ts_version(void);

/* ------------------------------------------------------------------------
 * Measurement support (not part of the FFN operation).
 */

/*
 * Per-kernel timing.  While enabled, every ts_* call records a HIP event
 * pair around each kernel it launches, on the call's stream.  ts_prof_read
 * synchronises on the recorded events and returns, for the kernel named
 * `kernel` ("ffn_main", "ffn_reduce", "ffn_gate_up", "ffn_down",
 * "ffn_topk_select", "ffn_topk_down", "ffn_given", "given_counts", "ffn_stats", "ffn_union",
 * "moe_router", "batch_prep", "batch_gate_up", "batch_down",
 * "batch_reduce", "batch_stats", "batch_union", "probe_read",
 * "probe_copy"), the number of launches and their summed duration in
 * milliseconds since the last ts_prof_reset.  Returns TS_ERR_HIP on a
 * HIP failure, TS_ERR_NULL for a NULL output pointer.  Not thread-safe.
 */
void ts_prof_enable(int on);
void ts_prof_reset(void);
ts_status ts_prof_read(const char *kernel, long *launches, double *total_ms);

/*
 * HBM probes.  ts_probe_read streams `bytes` (multiple of 16) from `src` and
 * writes one float per workgroup into `sink` (at least 4096 floats); it
 * measures the achievable read bandwidth.  ts_probe_copy copies `bytes`
 * (multiple of 16) from src to dst; its HBM counter readings calibrate the
 * traffic counters against a transfer of known size.
 */
ts_status ts_probe_read(const void *src, size_t bytes, float *sink, void *stream);
ts_status ts_probe_copy(const void *src, void *dst, size_t bytes, void *stream);

/*
 * Tuning knobs (process-wide; 0 restores the default).  Keys:
 *   "ffn_tile"   neurons per workgroup of the single-token kernels (4..128,
 *                multiple of 4; the fused kernel caps it at 64)
 *   "ffn_path"   0 = pipelined single-token kernel, 1 = split gate+up /
 *                down, 2 = fused single-token kernel
 *   "batch_path" 0 = matrix-core batched path for batch > 1 (bf16),
 *                1 = single-token kernels per token
 *   "gate_tile"  neurons per workgroup of the split path's gate+up kernel
 *                (4..64, multiple of 4)
 *   "down_chunks" tile groups per slot in the split path's down kernel, and
 *                per group in the batched down kernel
 *   "rif"        weight rows in flight per wave in the row dot products
 *                (1 or 2)
 *   "bx_gate"    batched gate+up kernel: 0 default (8 token slots per
 *                group: one 32-row tile per workgroup, k-steps of 32 per
 *                batch x batches in flight 2 x 2; 16 or more: two 32-row
 *                tiles per workgroup, 2 x 2); for 8 slots 1 = 2 x 2,
 *                2 = 2 x 4; for 16 slots 1 = 2 x 2 and 2 = 2 x 4 on one
 *                tile per workgroup; 3 = one tile per workgroup with its
 *                default load shape (4 x 2 at 16 slots, 2 x 2 past that)
 *   "bx_down"    batched down kernel for up to 32 tokens per group: 0 default
 *                (2 blocks of 32 rows in flight per wave), 1 = 3 blocks
 *   "bx_vgroup"  batched MoE layer: 0 default (token slots per expert group
 *                about twice the expected expert load; an expert with more
 *                tokens takes further groups), 1 = one group per expert
 *                with slots for the whole batch
 *   "bx_xtok"    batched MoE layer: 0 default (the router also writes
 *                each token's x as bf16 high / low parts and the gate+up
 *                kernel gathers its group's tokens from them: no dispatch
 *                kernel, one copy of x for all expert groups), 1 = a
 *                dispatch kernel builds per-group x fragments (as the
 *                batched FFN does)
 *   "ffn_interleave" single-token kernels: 0 default (workgroup t takes
 *                neurons t, t + T, t + 2 T, ... of T workgroups per token,
 *                so the grid streams one narrow band of each matrix at a
 *                time; used while a matrix is below 2 GB and inter <=
 *                131072), 1 = contiguous tiles of neurons
 * Returns TS_ERR_SHAPE for an unknown key or out-of-range value.
 */
ts_status ts_tune_set(const char *key, int value);

#ifdef __cplusplus
}
#endif

#endif /* TURBOSPARSE_H */
