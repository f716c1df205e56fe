/*
 * sekv.h -- C ABI of the SeKV decode-step library for AMD Instinct MI355X (gfx950).
 *
 * One decode step of SeKV (Abaskohi, Carenini, West, He: "SeKV: Resolution-Adaptive
 * KV Cache with Hierarchical Semantic Memory for Long-Context LLM Inference"),
 * for one attention layer, on one GPU:
 *
 *   1. routing: score every span of every sequence for every query head against the
 *      span's coarse mean key (Sec. 3.2, eq. routing_gate, read with an identity
 *      projection: score = scale * q.k_bar_S + ln|S|);
 *   2. selection: per (sequence, KV head) keep the top_k spans in decreasing score
 *      (Sec. 3.3, budget rule), the key of a span being the largest score over the
 *      KV head's query heads; ties go to the lower span index;
 *   3. zoom-in: rebuild the selected spans' keys and values from their low-rank
 *      factors, K_hat = U diag(sigma) V^T (eq. key_reconstruction, gates folded into
 *      sigma), in registers/LDS only -- reconstructed tokens never reach HBM;
 *   4. one softmax over the mixed-resolution memory (Sec. 3.3): anchor tokens at full
 *      resolution, one coarse entry (k_bar, v_bar, score + ln|S|) per unselected span,
 *      and the reconstructed tokens of the selected spans.
 *
 * Conventions
 *   - Every pointer in sekv_cache, and every sel/logits/out/workspace pointer, is a
 *     DEVICE pointer owned by the caller.  Data arrays (q, anchors, summaries, factor
 *     arena) are 16-byte aligned, out 8-byte; sel, logits and the tables n_anchors,
 *     n_spans, span_len 4-byte; span_logsize and block_off 8-byte (the tiered step reads the
 *     factor arena from pinned host memory instead).  The step calls allocate nothing;
 *     only the set-up calls (sekv_graph_create, sekv_tier_create) do.
 *   - Calls enqueue work on the caller's stream and return; results are valid in
 *     stream order.  Calls never synchronise the device unless documented.
 *   - Errors found on the host (null or misaligned pointers, unsupported sizes, a small
 *     workspace) are returned before anything is enqueued.  HIP launch failures return
 *     SEKV_ERR_HIP.  sekv_last_error() gives a thread-local message for the last failure.
 *   - Device-side tables must satisfy n_anchors[b] <= max_anchors, n_spans[b] <=
 *     max_spans, 1 <= span_len <= max_span_len, every block inside the factor arena.
 *     The kernels clamp counts and skip out-of-arena blocks (flagging the workspace
 *     error word), so a bad table gives a wrong answer, never an out-of-bounds access.
 *   - Results are bitwise deterministic: fixed reduction order, no floating-point atomics.
 *   - Concurrent calls must use distinct workspaces; calls sharing a workspace must be
 *     ordered on one stream.  The library remembers, per workspace address, the shapes of
 *     the last call it enqueued there, and enqueues a zeroing kernel before a call whose
 *     shapes (hence workspace layout) differ.  Calls recorded into a caller's own stream
 *     capture are tracked at capture time, so such a graph must be replayed in the order
 *     it was captured relative to eager calls on the same workspace.
 *   - Forward progress does not depend on how many workgroups are resident.  Each routing
 *     chunk is claimed (an atomic exchange on a per-chunk workspace word) by the first
 *     workgroup to reach it: its own workgroup, or a workgroup whose share item has waited
 *     for it for a while and then computes every unclaimed chunk of its pair itself.  A
 *     share item therefore only ever waits for chunks that a running workgroup holds, and
 *     such a workgroup never waits, so a step completes even while other kernels hold most
 *     of the device.  The learned-routing kernel has no waits at all.
 */
#ifndef SEKV_H
#define SEKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SEKV_API __attribute__((visibility("default")))

typedef enum {
    SEKV_OK = 0,
    SEKV_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, inconsistent sizes      */
    SEKV_ERR_UNSUPPORTED = 2,   /* head_dim, rank, group size or top_k not supported */
    SEKV_ERR_WORKSPACE = 3,     /* workspace too small or not initialised            */
    SEKV_ERR_HIP = 4            /* a HIP runtime call failed; see sekv_last_error()  */
} sekv_status;

typedef enum { SEKV_F32 = 0, SEKV_BF16 = 1 } sekv_dtype;

/* Implementation choice for the zoomed spans (sekv_dims.flags bits 0..1). */
#define SEKV_ZOOM_DEFAULT 0     /* library default (currently FACTORED)                     */
#define SEKV_ZOOM_FACTORED 1    /* q.K_hat = U (sigma * (V^T q)), sum p V_hat = ((p^T U) sigma) V^T */

/* Shapes and types of one layer's decode step.  Validated on the host before any launch. */
typedef struct {
    int32_t batch;          /* B >= 0 sequences                                          */
    int32_t n_q_heads;      /* Hq; query head h reads KV head h / (Hq / Hkv)             */
    int32_t n_kv_heads;     /* Hkv; Hq / Hkv in {1, 2, 4, 8}                             */
    int32_t head_dim;       /* d in {64, 128}                                            */
    int32_t rank;           /* r: factor rank, one of 8, 16, 32, 64                      */
    int32_t top_k;          /* k: spans expanded per (sequence, KV head), 0 <= k <= 64   */
    int32_t max_anchors;    /* A_max >= 0: row stride of the anchor arrays               */
    int32_t max_spans;      /* M_max >= 1: row stride of the span arrays                 */
    int32_t max_span_len;   /* L_max >= 1: longest span                                  */
    int32_t dtype;          /* sekv_dtype of q, anchors, summaries and factors           */
    int32_t out_dtype;      /* sekv_dtype of out (F32 is allowed for BF16 storage)       */
    int32_t flags;          /* bits 0..1: SEKV_ZOOM_*; other bits must be zero           */
    double softmax_scale;   /* multiplies q.k everywhere, including the routing score    */
} sekv_dims;

/* The stored cache of one layer.  All device pointers, caller-owned.
 *   q            [B][Hq][d]
 *   anchor_k/v   [B][Hkv][A_max][d]       rows >= n_anchors[b] are ignored
 *   n_anchors    int32 [B]                full-resolution tokens (anchors + local window)
 *   sum_k/sum_v  [B][Hkv][M_max][d]       coarse mean key/value of each span
 *   n_spans      int32 [B]
 *   span_len     int32 [B][M_max]         |S| of span S of sequence b
 *   span_logsize double [B][M_max]        ln|S|, computed once by the caller
 *   factors      byte arena of span blocks, factors_bytes long
 *   block_off    int64 [B][Hkv][M_max]    byte offset of block (b, g, S); multiple of 16
 *   block_rank   int32 [B][Hkv][M_max] or NULL: retained ranks r_K | r_V << 16 of block
 *                (b, g, S); NULL means r_K = r_V = dims.rank for every block
 * A span block holds, in the storage dtype and in this order,
 *   U_K[|S|][r_K] | sigma_K[r_K] | Vt_K[r_K][d] | U_V[|S|][r_V] | sigma_V[r_V] | Vt_V[r_V][d]
 * i.e. the per-span factors of Sec. 3.2 (U, Sigma, V^T for keys, then for values), each
 * side keeping its own number of components after the deployment-time drop of the
 * components with negligible gates (eqs. rank_gates and key_reconstruction; the kept
 * gates are folded into sigma).  Ranks are multiples of 16 / element bytes (8 for bf16, 4
 * for f32) in [that, dims.rank]; a block with another rank is skipped and flagged like a
 * block outside the arena. */
typedef struct {
    const void *q;
    const void *anchor_k;
    const void *anchor_v;
    const int32_t *n_anchors;
    const void *sum_k;
    const void *sum_v;
    const int32_t *n_spans;
    const int32_t *span_len;
    const double *span_logsize;
    const void *factors;
    int64_t factors_bytes;
    const int64_t *block_off;
    const int32_t *block_rank;
} sekv_cache;

/* Human-readable name of a status code (static storage). */
SEKV_API const char *sekv_status_string(sekv_status status);

/* Thread-local message describing the last failing call on this thread ("" if none). */
SEKV_API const char *sekv_last_error(void);

/* Diagnostic phase trace.  In a library built with SEKV_PHASE_TRACE (libsekv_trace.so),
 * attaches a device buffer to the calling thread: every later step launch on this thread
 * whose work items fit writes, per item i, 16 int64 words at buf[16 i]: word 0 =
 * kind (0 routing item, 1 share item) << 60 | XCC id << 48 | workgroup index, words 1..12 =
 * the device's 100 MHz real-time counter at the item's phase marks (start, end, then
 * kind-specific marks; see sekv_step.h), 0 where a mark was not reached.  Launches whose
 * items do not fit in `bytes` are not traced.  buf == NULL detaches.  The product build
 * (libsekv.so) returns SEKV_ERR_UNSUPPORTED and never traces. */
SEKV_API sekv_status sekv_phase_trace(void *buf, size_t bytes);

/* Host-only validation of a sekv_dims; SEKV_OK if every library call accepts it. */
SEKV_API sekv_status sekv_check_dims(const sekv_dims *dims);

/* Bytes of device workspace the calls below need for these dims (0 if dims are invalid). */
SEKV_API size_t sekv_workspace_size(const sekv_dims *dims);

/* Zero a workspace on `stream`.  Required once before the first call that uses it; every
 * call leaves its counters zeroed again on completion.  ws: device, 256-byte aligned. */
SEKV_API sekv_status sekv_workspace_init(void *ws, size_t ws_bytes, hipStream_t stream);

/* Read and clear the workspace's device error word (synchronises `stream`).  Bits:
 * 1 = a wait for a selection timed out, 2 = a factor block lay outside the arena or its
 * rank-table entry was invalid, 4 = a selected index was out of range (sekv_build_cache:
 * an anchor index or span outside the sequence's tokens).  0 after every correct call. */
SEKV_API sekv_status sekv_workspace_status(void *ws, size_t ws_bytes, hipStream_t stream,
                                  int32_t *error_bits);

/* Steps 1-2 (routing and selection; Sec. 3.2 eq. routing_gate, Sec. 3.3 budget rule).
 *   sel    out, int32 [B][Hkv][top_k]: spans in decreasing key order, -1 past n_spans[b]
 *   logits out, float [B][Hq][M_max] or NULL: the routing scores (score, not sigmoid);
 *          entries past n_spans[b] are -inf.
 * Reads q, sum_k, n_spans, span_logsize. */
SEKV_API sekv_status sekv_route_topk(const sekv_dims *dims, const sekv_cache *cache, int32_t *sel,
                            float *logits, void *ws, size_t ws_bytes, hipStream_t stream);

/* Steps 3-4 for a given selection (Sec. 3.3, mixed-resolution attention).
 *   sel    in, int32 [B][Hkv][top_k] as produced by sekv_route_topk (-1 = empty slot)
 *   logits in, float [B][Hq][M_max] routing scores, or NULL to recompute them from sum_k
 *   out    out, [B][Hq][d] in out_dtype */
SEKV_API sekv_status sekv_zoom_attend(const sekv_dims *dims, const sekv_cache *cache, const int32_t *sel,
                             const float *logits, void *out, void *ws, size_t ws_bytes,
                             hipStream_t stream);

/* Steps 1-4 fused into one launch: sel and out as above; the routing scores stay in the
 * workspace.  Summary rows are read once (keys for routing, values for the coarse
 * entries in the same pass). */
SEKV_API sekv_status sekv_decode_step(const sekv_dims *dims, const sekv_cache *cache, int32_t *sel,
                             void *out, void *ws, size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): sekv_decode_step with its workspace
 * in a static device array the library holds on every device it runs on, until the
 * process ends (SEKV_NOALLOC_MAX_WORKSPACE bytes per device).  Allocates nothing: the
 * first call on a device looks up the array's address there; the caller passes inputs
 * and outputs as for sekv_decode_step.  Shapes whose sekv_workspace_size exceeds the
 * array are refused with SEKV_ERR_WORKSPACE.  Every call on a device shares that
 * device's array: calls that may overlap on one device (several streams or threads)
 * race and give wrong results; order them on one stream.  The array keeps the last
 * call's contents; the library zeroes it (a kernel on `stream`) on its first use and
 * whenever the shapes change.  sekv_workspace_status cannot read this array; a
 * device-side wait timeout or out-of-arena block is not reported. */
#define SEKV_NOALLOC_MAX_WORKSPACE (16u << 20)
SEKV_API sekv_status sekv_decode_step_noalloc(const sekv_dims *dims, const sekv_cache *cache,
                                              int32_t *sel, void *out, hipStream_t stream);

/* ----------------------------------------------------------------------------------
 * The paper's own selection rule (learned routing).  In place of steps 1-2 above:
 *   q'_h = W_h q_h                                  (Sec. 3.2 eq. query_projection)
 *   x_h,S = q'_h . Kbar_h,S / sqrt(d') + ln|S|      (eq. routing_gate, before the sigmoid)
 *   query head h votes for span S when x_h,S > ln(tau_h / (1 - tau_h)), i.e. when the
 *   gate sig(x_h,S) exceeds its threshold tau_h       (Sec. 3.3 eq. zoom_decision)
 * A span is expanded for its (sequence, KV head) when a query head of the group votes for
 * it; voted spans are taken in decreasing order of their largest voting gate (ties to the
 * lower span index) while the expanded tokens stay within budget_tokens and the count
 * within top_k (the budget cap of Sec. 3.3); the expanded spans serve every query head of
 * the group.  The selection is exact: q' is summed over d in float64 in index order and
 * rounded once to float32, the gate's dot product is summed over d' in float64 in index
 * order, then x = (s * (1/sqrt(d'))) + ln|S| with two roundings (1/sqrt(d') computed in
 * float64 as 1.0 / sqrt(d')).
 * ---------------------------------------------------------------------------------- */
typedef struct {
    int32_t route_dim;          /* d': multiple of 8, 8 <= d' <= 64                        */
    int32_t reserved;           /* must be 0                                               */
    int64_t budget_tokens;      /* >= 0: expanded tokens allowed per (sequence, KV head)   */
    const void *proj;           /* device [Hq][d'][d], storage dtype: W of each query head */
    const void *sum_route;      /* device [B][Hq][M_max][d'], storage dtype: routing
                                   summaries (normalised, eq. summary_key); rows past
                                   n_spans[b] are ignored                                  */
    const double *thresholds;   /* device double [Hq]: ln(tau_h / (1 - tau_h))             */
} sekv_gate;

/* Selection under the learned rule.  Reads q, n_spans, span_len, span_logsize (not the
 * factors or the summaries' keys/values) and the gate arrays; proj and sum_route 16-byte
 * aligned, thresholds and gate_logits 8-byte.
 *   sel          out, int32 [B][Hkv][top_k]: expanded spans in expansion order, -1 after
 *   gate_logits  out, double [B][Hq][M_max] or NULL: x_h,S (-inf past n_spans[b]);
 *                the gate itself is sig(x)
 * One launch, no wait between workgroups; uses its own section of the workspace. */
SEKV_API sekv_status sekv_route_gated(const sekv_dims *dims, const sekv_cache *cache,
                                      const sekv_gate *gate, int32_t *sel, double *gate_logits,
                                      void *ws, size_t ws_bytes, hipStream_t stream);

/* One decode step under the learned rule: sekv_route_gated, then sekv_zoom_attend with
 * that selection (coarse entries of unexpanded spans use scale * q.k_bar + ln|S|, as in
 * the step above).  Two launches on `stream`. */
SEKV_API sekv_status sekv_decode_step_gated(const sekv_dims *dims, const sekv_cache *cache,
                                            const sekv_gate *gate, int32_t *sel, void *out,
                                            void *ws, size_t ws_bytes, hipStream_t stream);

/* ----------------------------------------------------------------------------------
 * Prefill-side builder: the step before the decode path.  From a layer's token keys and
 * values and the tokens' surprisal H_t (produced by the prefill forward pass, Sec. 3.1),
 * build the stored cache the calls above read.
 *   1. sekv_segment: boundaries where H_t > mu + alpha sigma (mu, sigma: mean and
 *      population standard deviation of the sequence's surprisal, Sec. 3.1), each sum
 *      formed in one fixed order -- 1024 partial sums, partial j adding tokens j, j + 1024,
 *      ... in float64, then combined by halving (j += j + h for h = 512, ..., 1) -- and
 *      threshold mu + (alpha * sigma) without fused multiply-add, so the decisions are
 *      exact.  Anchors: the boundary tokens, the last `window` tokens, and the tokens of
 *      any run between neighbouring anchors shorter than `min_span`; spans: the other runs.
 *   2. sekv_build_layout (host only): block offsets and ranks of the factor arena.
 *   3. sekv_build_cache: anchor rows, surprisal-weighted mean key/value of each span
 *      (eq. surprisal_weight), |S|, ln|S|, and each span's factors for keys and values by
 *      a randomized truncated SVD of rank r = min(|S|, d, R_max) (eq. key_svd), stored with
 *      the rank rounded up to 16 / element bytes (extra components zero; block_rank).
 *      The SVD sketches the span with the caller's d x l Gaussian test matrix; each
 *      subspace iteration (`power`) sketches it again with an orthonormal basis of the
 *      previous pass's dominant row space, which sharpens the captured subspace when the
 *      spectrum is flat (a span of at most `sketch` tokens needs none and gets none).
 *      Directions of the sketch below 1e-8 of its largest Gram diagonal entry are dropped
 *      (rank-deficient spans), as are components below 1e-5 of the largest singular value.
 * ---------------------------------------------------------------------------------- */
typedef struct {
    int32_t batch;          /* B >= 0                                                        */
    int32_t n_kv_heads;     /* Hkv >= 1                                                      */
    int32_t head_dim;       /* d in {64, 128}                                                */
    int32_t max_tokens;     /* N_max >= 1: row stride of the token arrays                    */
    int32_t rank;           /* R_max: multiple of 16 / element bytes, at most 40 and sketch   */
    int32_t sketch;         /* l: columns of the random test matrix, even, R_max <= l <= 40   */
    int32_t min_span;       /* L_min >= 2                                                    */
    int32_t window;         /* w >= 0                                                        */
    int32_t sweeps;         /* Jacobi sweeps of the small eigenproblems, 1..32 (8 is ample)   */
    int32_t dtype;          /* sekv_dtype of keys, values and the built cache                */
    int32_t power;          /* subspace iterations of the randomized SVD, 0..4 (1 is usual)   */
    int32_t reserved;       /* 0                                                             */
    double alpha;           /* boundary sensitivity                                          */
} sekv_build_dims;

/* Scratch bytes sekv_segment needs (device, 16-byte aligned; no initialisation needed). */
SEKV_API size_t sekv_segment_workspace_size(const sekv_build_dims *dims);

/* Segmentation.  All device pointers: surprisal float [B][N_max], n_tokens int32 [B] (values
 * are clamped to [0, N_max]); out: n_anchors [B], anchor_idx [B][N_max] (token indices,
 * ascending), n_spans [B], span_start [B][N_max], span_len [B][N_max] (token order).  One
 * workgroup per sequence. */
SEKV_API sekv_status sekv_segment(const sekv_build_dims *dims, const float *surprisal,
                                  const int32_t *n_tokens, int32_t *n_anchors, int32_t *anchor_idx,
                                  int32_t *n_spans, int32_t *span_start, int32_t *span_len, void *ws,
                                  size_t ws_bytes, hipStream_t stream);

/* Host only: the factor arena of a segmentation read back to the host.  n_spans [B] and
 * span_len [B][N_max] are the segmentation's; max_spans >= every n_spans[b].  Writes
 * block_off [B][Hkv][max_spans] (256-byte aligned blocks in (b, g, S) order) and
 * block_rank [B][Hkv][max_spans] (r_S | r_S << 16, 0 past n_spans[b]); returns the arena
 * bytes, or -1 with sekv_last_error() set. */
SEKV_API int64_t sekv_build_layout(const sekv_build_dims *dims, int32_t max_spans, const int32_t *n_spans,
                                   const int32_t *span_len, int64_t *block_off, int32_t *block_rank);

/* The cache.  Device pointers: keys/values [B][Hkv][N_max][d], surprisal, n_tokens and the
 * segmentation arrays as above, omega float [d][sketch] (the random test matrix, drawn by
 * the caller), block_off/block_rank from sekv_build_layout (copied to the device).
 * Outputs, laid out as sekv_cache: anchor_k/v [B][Hkv][max_anchors][d] (rows past
 * n_anchors[b] untouched), sum_k/v [B][Hkv][max_spans][d], span_len [B][max_spans],
 * span_logsize [B][max_spans], the factor arena (factors_bytes).  max_anchors and
 * max_spans must cover every n_anchors[b] and n_spans[b] (larger counts are clamped).
 * Anchor indices and spans must lie in [0, n_tokens[b]) (n_tokens clamped to [0, N_max]);
 * an anchor row or span outside it is skipped.
 * ws: a step workspace of at least 256 bytes whose error word reports blocks outside the
 * arena (bit 2) and skipped anchor rows or spans (bit 4). */
SEKV_API sekv_status sekv_build_cache(const sekv_build_dims *dims, const void *keys, const void *values,
                                      const float *surprisal, const int32_t *n_tokens,
                                      const int32_t *n_anchors, const int32_t *anchor_idx,
                                      const int32_t *n_spans, const int32_t *span_start,
                                      const int32_t *span_len_seg, const float *omega,
                                      int32_t max_anchors, int32_t max_spans, void *anchor_k,
                                      void *anchor_v, void *sum_k, void *sum_v, int32_t *span_len,
                                      double *span_logsize, void *factors, int64_t factors_bytes,
                                      const int64_t *block_off, void *ws, size_t ws_bytes,
                                      hipStream_t stream);

/* ----------------------------------------------------------------------------------
 * Several layers in one HIP graph.  A decode step of an L-layer model runs the step
 * above once per layer (each attention layer keeps its own span cache, Sec. 3.2; the
 * per-layer cost analysis of App. D sums over layers).  sekv_graph_create validates
 * every layer and captures one sekv_decode_step per layer, in layer order, into an
 * executable HIP graph; sekv_graph_launch replays it on any stream.
 *   layers  host array [n_layers] of sekv_cache (device pointers as above); every
 *           layer has the shapes of `dims`
 *   sel     device int32 [n_layers][B][Hkv][top_k], may be NULL when top_k == 0
 *   out     device [n_layers][B][Hq][d] in out_dtype
 *   ws      one workspace for all layers (the launches run one after another)
 * The graph keeps the pointers it was created with: the caller keeps every buffer
 * alive and in place until sekv_graph_destroy.  Launches of one graph, or of graphs
 * and calls sharing its workspace, must be ordered (one stream); concurrent replays
 * race on the workspace.  The handle is host memory owned by the library; the graph
 * itself records only kernel launches.
 * -------------------------------------------------------------------------------- */
typedef struct sekv_graph sekv_graph;

SEKV_API sekv_status sekv_graph_create(const sekv_dims *dims, const sekv_cache *layers,
                                       int32_t n_layers, int32_t *sel, void *out, void *ws,
                                       size_t ws_bytes, sekv_graph **graph);

/* Enqueue one replay of the graph (all layers) on `stream`. */
SEKV_API sekv_status sekv_graph_launch(sekv_graph *graph, hipStream_t stream);

/* Free the graph and its handle (NULL is a no-op).  No replay may be pending. */
SEKV_API sekv_status sekv_graph_destroy(sekv_graph *graph);

/* ----------------------------------------------------------------------------------
 * Pinned-host tier.  The paper keeps every span's low-rank factors in CPU memory and
 * moves only the zoomed spans' factors to the GPU at each step, overlapped with the
 * rest of the step (Sec. 3.2, last paragraph; App. D: the per-step transfer is the
 * sum over the zoomed spans of 2 H_kv r (|S| + d_h + 1) elements, independent of the
 * context length).  Here anchors, summaries and span tables stay in HBM and the factor
 * arena lives in pinned host memory.
 *
 * sekv_decode_step_tiered, per sequence b in order:
 *   1. routing and selection of b on `main` (steps 1-2);
 *   2. the selected blocks of b move from the pinned arena to the tier's device staging
 *      area on `side`, after an event on b's selection:
 *        SEKV_TIER_GATHER: one kernel reads b's selection and tables on the device and
 *          copies each selected block, through the arena's device mapping, to the fixed
 *          staging slot of its selection slot.  Nothing waits on the host: the call only
 *          enqueues work, and can be captured in a graph.
 *        SEKV_TIER_MEMCPY: the selection is read back to a pinned mirror; the host waits
 *          for b's selection, packs its blocks in arena order and issues one
 *          hipMemcpyAsync per run of blocks that are neighbours in the arena, then the
 *          staging offset table of b (hipMemcpyAsync).
 *   3. `main` waits for those copies (an event) and runs steps 3-4 of b from staging.
 * Copies of sequence b overlap the routing of later sequences and the attention of
 * earlier ones.  Results are those of sekv_route_topk followed by sekv_zoom_attend with
 * the routing scores, on a device-resident copy of the arena, in both modes.
 * -------------------------------------------------------------------------------- */

/* The factor arena in pinned host memory (hipHostMalloc), and host copies of the span
 * tables the host needs to address it. */
typedef struct {
    const void *arena;              /* pinned host bytes, span blocks as in sekv_cache       */
    int64_t arena_bytes;
    const int64_t *block_off;       /* host int64 [B][Hkv][M_max]: byte offset of each block */
    const int32_t *span_len;        /* host int32 [B][M_max]: |S|                            */
    const int32_t *block_rank;      /* host int32 [B][Hkv][M_max] r_K | r_V << 16, or NULL
                                       (then cache->block_rank must be NULL too)             */
} sekv_host_factors;

typedef struct sekv_tier sekv_tier;

/* How a tier moves the selected blocks (see above). */
typedef enum { SEKV_TIER_GATHER = 0, SEKV_TIER_MEMCPY = 1 } sekv_tier_copy;

/* Set-up (allocates): pinned mirrors of the selection and of the staging offsets,
 * device staging for batch * Hkv * top_k blocks of max_span_len tokens, a routing-score
 * buffer, copy counters and events, on the current device.  copy_mode is a
 * sekv_tier_copy.  dims is copied; every step must pass identical dims. */
SEKV_API sekv_status sekv_tier_create(const sekv_dims *dims, int32_t copy_mode, sekv_tier **tier);

/* Free everything the tier holds (NULL is a no-op).  No step may be pending. */
SEKV_API sekv_status sekv_tier_destroy(sekv_tier *tier);

/* Device staging bytes the tier holds (0 for NULL). */
SEKV_API size_t sekv_tier_staging_size(const sekv_tier *tier);

/* Host-link figures of the last tiered step: bytes moved host to device, number of
 * copies (runs of neighbouring blocks for SEKV_TIER_MEMCPY, blocks for SEKV_TIER_GATHER),
 * and the time on the side stream from the first copy's start (gather: from the first
 * sequence's selection) to the last copy's end.  Valid once that step has completed;
 * in gather mode the call reads the device's counters (a synchronous copy). */
SEKV_API sekv_status sekv_tier_last_copy(sekv_tier *tier, int64_t *bytes, int32_t *copies,
                                         float *ms);

/* One decode step with the factors in pinned host memory.
 *   cache   device arrays as for sekv_decode_step; cache->factors is not read; in gather
 *           mode cache->block_off is a device copy of host->block_off (offsets into the
 *           host arena), in memcpy mode it is not read
 *   host    the pinned arena and host tables; an arena that is not pinned (gather mode:
 *           pinned and device-mapped) memory is an SEKV_ERR_INVALID_ARG; a selected block
 *           outside the arena is an SEKV_ERR_INVALID_ARG in memcpy mode, and in gather
 *           mode is skipped with the workspace error bit 2 set
 *   sel     device int32 [B][Hkv][top_k]; out device [B][Hq][d] in out_dtype
 *   ws      workspace of sekv_workspace_size(dims)
 *   main    stream of the kernels; side: stream of the host-to-device copies (both at the
 *           default priority; side must differ from main for the overlap)
 * The tier must not be shared by concurrent steps. */
SEKV_API sekv_status sekv_decode_step_tiered(const sekv_dims *dims, const sekv_cache *cache,
                                             const sekv_host_factors *host, sekv_tier *tier,
                                             int32_t *sel, void *out, void *ws, size_t ws_bytes,
                                             hipStream_t main, hipStream_t side);

/* Several layers of one decode step with the factors in pinned host memory, and the
 * cross-layer prefetch of the paper's pipelined transfer (Sec. 3.2, last paragraph: the
 * GPU computation overlaps the CPU-GPU transfer of the selected bases).  Span boundaries
 * come from the sequence's surprisal (Sec. 3.1), so every layer has the same spans; a
 * span zoomed by layer l is a likely zoom of layer l + 1.  Per layer l, in order:
 *   1. routing and selection of every sequence on `main`, after layer l - 1's attention
 *      (in a model, layer l's queries need layer l - 1's output);
 *   2. on `side`, after an event on that selection: every selected block of layer l that
 *      is not already in the layer's staging is copied there through the arena's device
 *      mapping (the "miss" copies, on the critical path);
 *   3. with prefetch = 1, still on `side`: layer l + 1's blocks of the spans layer l
 *      selected are copied into layer l + 1's staging, overlapping layer l's attention
 *      and layer l + 1's routing (the speculative copies, off the critical path);
 *   4. `main` waits for step 2 and runs layer l's attention from staging.
 * Layers alternate between two staging buffers, each a prefetch region and a miss region
 * of batch * Hkv * top_k slots; the tier allocates them on the first call (2 x 2 x the
 * staging of sekv_tier_staging_size, plus offset tables).  Results are bit for bit those
 * of sekv_decode_step_tiered layer by layer, with or without prefetch.
 *   dims      as for sekv_decode_step_tiered (identical to the tier's; every layer has them)
 *   caches    n_layers device caches (cache.factors not read; cache.block_off is the
 *             device copy of the host offsets, as in gather mode)
 *   hosts     n_layers pinned, device-mapped host arenas and tables
 *   sel       device int32 [n_layers][B][Hkv][top_k]; out device [n_layers][B][Hq][d]
 * The tier must be a SEKV_TIER_GATHER tier.  A selected block outside its arena is skipped
 * with the workspace error bit 2 set. */
SEKV_API sekv_status sekv_decode_layers_tiered(const sekv_dims *dims, const sekv_cache *caches,
                                               const sekv_host_factors *hosts, int32_t n_layers,
                                               int32_t prefetch, sekv_tier *tier, int32_t *sel,
                                               void *out, void *ws, size_t ws_bytes, hipStream_t main,
                                               hipStream_t side);

/* Copy counters of the last sekv_decode_layers_tiered call, over all its layers:
 * stats[0] bytes and stats[1] blocks copied after a selection (the critical path),
 * stats[2] bytes and stats[3] blocks prefetched.  Valid once that call has completed
 * (a synchronous read of the device counters). */
SEKV_API sekv_status sekv_tier_layer_stats(sekv_tier *tier, int64_t stats[4]);

/* Debug check of the device-side preconditions of the step calls, made on HOST copies of
 * a cache (every pointer in host_copy is a host pointer; factors_bytes is the arena
 * size), so it is slow and synchronous.  Checks, for every sequence b:
 *   0 <= n_anchors[b] <= max_anchors, 0 <= n_spans[b] <= max_spans, n_anchors[b] +
 *   n_spans[b] >= 1; 1 <= span_len <= max_span_len and span_logsize = ln(span_len) for
 *   every span; every span's block 16-byte aligned and inside the arena (when top_k > 0),
 *   with valid ranks when the cache has a rank table;
 *   every stored value of q, the anchors, the summaries and the factor blocks finite.
 * Returns SEKV_OK, or SEKV_ERR_INVALID_ARG with the first violation in sekv_last_error(). */
SEKV_API sekv_status sekv_validate_cache(const sekv_dims *dims, const sekv_cache *host_copy);

#ifdef __cplusplus
}
#endif

#endif /* SEKV_H */
