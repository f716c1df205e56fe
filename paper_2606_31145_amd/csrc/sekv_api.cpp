// C ABI of the SeKV decode-step library: host-side validation, workspace layout and
// launch set-up.  Every check that can be made on the host is made here, before
// anything is enqueued; the kernels clamp device-side table values on their own.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "sekv.h"
#include "sekv_host.h"
#include "sekv_internal.h"

namespace {

using sekv::fail;

// Diagnostic phase-trace buffer attached by sekv_phase_trace (trace builds only).
thread_local int64_t *g_trace = nullptr;
thread_local size_t g_trace_bytes = 0;

}  // namespace

namespace sekv {
int64_t *trace_buffer(size_t *bytes) {
    *bytes = g_trace_bytes;
    return g_trace;
}
}  // namespace sekv

namespace {

sekv_status hip_fail(hipError_t e, const char *what) {
    return fail(SEKV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

sekv_status check_dims_impl(const sekv_dims *d) { return sekv::check_dims(d); }
sekv_status check_cache(const sekv_dims *d, const sekv_cache *c, bool need_factors) {
    return sekv::check_cache(d, c, need_factors);
}

sekv_status check_ws(const sekv_dims *d, void *ws, size_t ws_bytes) {
    const size_t need = sekv_workspace_size(d);
    if (!ws) return fail(SEKV_ERR_WORKSPACE, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(ws) & 255u)
        return fail(SEKV_ERR_WORKSPACE, "workspace not 256-byte aligned");
    if (ws_bytes < need)
        return fail(SEKV_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
    return SEKV_OK;
}

// Per-device cache of the resident-workgroup count of each kernel instantiation.
struct OccKey { int dev, dtype, d, g; };
std::mutex g_occ_mu;
struct OccEntry { OccKey k; int n; };
OccEntry g_occ[64];
int g_occ_n = 0;

int resident(int dtype, int head_dim, int group) {
    int dev = 0;
    (void)hipGetDevice(&dev);
    std::lock_guard<std::mutex> lk(g_occ_mu);
    for (int i = 0; i < g_occ_n; ++i) {
        const OccKey &k = g_occ[i].k;
        if (k.dev == dev && k.dtype == dtype && k.d == head_dim && k.g == group) return g_occ[i].n;
    }
    const int n = sekv::resident_workgroups(dtype, head_dim, group);
    if (g_occ_n < 64) g_occ[g_occ_n++] = {{dev, dtype, head_dim, group}, n};
    return n;
}

// Validate one call and fill its launch parameters.  *launch is false when there is
// nothing to run (empty batch, or no work items).
sekv_status prepare(int mode, const sekv_dims *d, const sekv_cache *c, int32_t *sel_out,
                    float *logits_out, const int32_t *sel_in, const float *logits_in, void *out,
                    void *ws, size_t ws_bytes, sekv::Params *pp, bool *launch) {
    *launch = false;
    sekv_status st = check_dims_impl(d);
    if (st != SEKV_OK) return st;
    st = check_cache(d, c, mode != sekv::kModeRoute);
    if (st != SEKV_OK) return st;
    st = check_ws(d, ws, ws_bytes);
    if (st != SEKV_OK) return st;
    if (d->batch == 0) return SEKV_OK;
    if (mode != sekv::kModeAttend && d->top_k > 0 && !sel_out)
        return fail(SEKV_ERR_INVALID_ARG, "sel is NULL");
    if (mode == sekv::kModeAttend && d->top_k > 0 && !sel_in)
        return fail(SEKV_ERR_INVALID_ARG, "sel is NULL");
    if (mode != sekv::kModeRoute && !out) return fail(SEKV_ERR_INVALID_ARG, "out is NULL");
    // element accesses: sel and logits 4-byte, out in pairs of values (8-byte)
    auto mis = [](const void *q, uintptr_t a) { return (reinterpret_cast<uintptr_t>(q) & (a - 1)) != 0; };
    if (mis(sel_out, 4) || mis(sel_in, 4) || mis(logits_out, 4) || mis(logits_in, 4) || mis(out, 8))
        return fail(SEKV_ERR_INVALID_ARG, "sel/logits not 4-byte or out not 8-byte aligned");

    const sekv::Shape s = sekv::make_shape(*d);
    const sekv::WsLayout L = sekv::make_layout(s);
    unsigned char *w = static_cast<unsigned char *>(ws);

    sekv::Params p{};
    p.mode = mode;
    p.B = s.B; p.Hq = s.Hq; p.Hkv = s.Hkv; p.r = s.r; p.k = s.k;
    p.A_max = s.A_max; p.M_max = s.M_max;
    p.n_rc = s.n_rc; p.kc = s.kc; p.n_cand = s.n_cand; p.n_zi = s.n_zi;
    // routing items run unless the caller hands in the routing scores; share items run
    // unless only the selection is asked for
    const bool scores = !(mode == sekv::kModeAttend && logits_in != nullptr);
    const int n_route = scores ? s.P * s.n_rc : 0;
    const int n_share = (mode == sekv::kModeRoute) ? 0 : s.P * s.n_zi;
    p.end_route = n_route;
    p.end_share = n_route + n_share;
    // Share items run slot-major after the routing items.  When the first round of items
    // ends inside the share items, the slots that start in it take all the anchors, and
    // the slots that start later (after a routing item) only select, zoom and fold
    // summaries.
    p.n_early = s.n_zi;
    const int first = sekv::kRoundItems - n_route;
    if (n_share > 0 && first >= s.P && first < n_share) p.n_early = first / s.P;
    p.out_f32 = d->out_dtype == SEKV_F32;
    p.zoom_impl = (d->flags & 3) == SEKV_ZOOM_DEFAULT ? SEKV_ZOOM_FACTORED : (d->flags & 3);
    p.scale = d->softmax_scale;
    p.scale_log2 = float(d->softmax_scale * 1.4426950408889634074);
    p.q = c->q; p.anchor_k = c->anchor_k; p.anchor_v = c->anchor_v; p.n_anchors = c->n_anchors;
    p.sum_k = c->sum_k; p.sum_v = c->sum_v; p.n_spans = c->n_spans; p.span_len = c->span_len;
    p.span_logsize = c->span_logsize;
    p.factors = static_cast<const unsigned char *>(c->factors);
    p.factors_bytes = c->factors_bytes;
    p.block_off = c->block_off;
    p.block_rank = c->block_rank;
    p.sel_out = sel_out; p.logits_out = logits_out; p.sel_in = sel_in; p.logits_in = logits_in;
    p.out = out;
    p.hdr = reinterpret_cast<sekv::WsHeader *>(w);
    p.route_cnt = reinterpret_cast<uint32_t *>(w + L.route_cnt);
    p.sel_ready = reinterpret_cast<uint32_t *>(w + L.sel_ready);
    p.part_cnt = reinterpret_cast<uint32_t *>(w + L.part_cnt);
    p.claim = reinterpret_cast<uint32_t *>(w + L.claim);
    p.zrec = reinterpret_cast<int4 *>(w + L.zrec);
    p.cand = reinterpret_cast<uint64_t *>(w + L.cand);
    p.tlg = reinterpret_cast<uint64_t *>(w + L.tlg);
    p.part_ml = reinterpret_cast<uint64_t *>(w + L.part_ml);
    p.part_o = reinterpret_cast<uint64_t *>(w + L.part_o);

    // Fused mode ranks the candidates inside every share item when they fit its LDS
    // buffer; otherwise one workgroup per pair merges them.
    const bool per_item = s.n_cand <= sekv::kMergeBuf;
    p.merger = (mode == sekv::kModeRoute) || (mode == sekv::kModeFused && !per_item);
    const int cap = resident(d->dtype, d->head_dim, s.G);
    p.grid = std::max(1, std::min(p.end_share, cap));
    p.trace = nullptr;
    if (g_trace && g_trace_bytes >= size_t(p.end_share) * sekv::kTraceSlots * sizeof(int64_t))
        p.trace = g_trace;
    *pp = p;
    *launch = p.end_share > 0;
    return SEKV_OK;
}

// ------------------------------------------------------------------------------------
// Workspace state.  A launch leaves its workspace ready for the next launch with the SAME
// layout (counters zero, epoch advanced).  Sections sit at offsets that depend on the
// shapes, so a launch with another layout could meet words that an earlier layout left
// there: stale counters, or untagged data in place of tagged words.  The library
// therefore remembers, per workspace address, the layout of the last launch it enqueued
// there (calls sharing a workspace are ordered on one stream, so enqueue order is
// execution order), and zeroes the whole workspace on the stream before a launch whose
// layout differs, before the 2^31-th launch since the last zeroing (the 32-bit epoch
// never wraps), and whenever it has no record (first use, or after eviction).
// ------------------------------------------------------------------------------------
std::mutex g_ws_mu;
sekv::WsTracker g_ws;

void ws_note_zeroed(void *ws, size_t bytes) {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    g_ws.zeroed(reinterpret_cast<uintptr_t>(ws), bytes);
}

hipError_t ws_prepare(void *ws, size_t ws_bytes, uint64_t key, uint64_t n_launch, hipStream_t stream) {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    if (g_ws.before_launch(reinterpret_cast<uintptr_t>(ws), ws_bytes, key, n_launch))
        return sekv::launch_zero(ws, ws_bytes & ~size_t(15), stream);
    return hipSuccess;
}

sekv_status run(int mode, const sekv_dims *d, const sekv_cache *c, int32_t *sel_out,
                float *logits_out, const int32_t *sel_in, const float *logits_in, void *out,
                void *ws, size_t ws_bytes, hipStream_t stream) {
    sekv::Params p{};
    bool launch = false;
    const sekv_status st = prepare(mode, d, c, sel_out, logits_out, sel_in, logits_in, out, ws,
                                   ws_bytes, &p, &launch);
    if (st != SEKV_OK || !launch) return st;
    hipError_t e = ws_prepare(ws, ws_bytes, sekv::layout_key(sekv::make_shape(*d)), 1, stream);
    if (e != hipSuccess) return hip_fail(e, "workspace zero kernel");
    e = sekv::launch_step(p, d->dtype, d->head_dim, d->n_q_heads / d->n_kv_heads, stream);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return SEKV_OK;
}

}  // namespace

namespace sekv {
sekv_status run_fused_step(const sekv_dims *d, const sekv_cache *c, int32_t *sel, void *out, void *ws,
                           size_t ws_bytes, hipStream_t stream) {
    return run(kModeFused, d, c, sel, nullptr, nullptr, nullptr, out, ws, ws_bytes, stream);
}
}  // namespace sekv

extern "C" {

const char *sekv_status_string(sekv_status status) {
    switch (status) {
        case SEKV_OK: return "SEKV_OK";
        case SEKV_ERR_INVALID_ARG: return "SEKV_ERR_INVALID_ARG";
        case SEKV_ERR_UNSUPPORTED: return "SEKV_ERR_UNSUPPORTED";
        case SEKV_ERR_WORKSPACE: return "SEKV_ERR_WORKSPACE";
        case SEKV_ERR_HIP: return "SEKV_ERR_HIP";
    }
    return "SEKV_ERR_UNKNOWN";
}

const char *sekv_last_error(void) { return sekv::last_error(); }

sekv_status sekv_check_dims(const sekv_dims *dims) { return check_dims_impl(dims); }

sekv_status sekv_phase_trace(void *buf, size_t bytes) {
#ifdef SEKV_PHASE_TRACE
    if (buf && (reinterpret_cast<uintptr_t>(buf) & 7))
        return fail(SEKV_ERR_INVALID_ARG, "trace buffer not 8-byte aligned");
    g_trace = static_cast<int64_t *>(buf);
    g_trace_bytes = buf ? bytes : 0;
    return SEKV_OK;
#else
    (void)buf;
    (void)bytes;
    return fail(SEKV_ERR_UNSUPPORTED, "phase tracing needs the library built with SEKV_PHASE_TRACE");
#endif
}

size_t sekv_workspace_size(const sekv_dims *dims) {
    char saved[512];
    std::snprintf(saved, sizeof(saved), "%s", sekv::last_error());
    const sekv_status st = check_dims_impl(dims);
    fail(SEKV_OK, "%s", saved);
    if (st != SEKV_OK) return 0;
    return sekv::make_layout(sekv::make_shape(*dims)).total;
}

sekv_status sekv_workspace_init(void *ws, size_t ws_bytes, hipStream_t stream) {
    if (!ws) return fail(SEKV_ERR_WORKSPACE, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(ws) & 255u)
        return fail(SEKV_ERR_WORKSPACE, "workspace not 256-byte aligned");
    if (ws_bytes % 16) return fail(SEKV_ERR_WORKSPACE, "workspace size not a multiple of 16");
    const hipError_t e = sekv::launch_zero(ws, ws_bytes, stream);
    if (e != hipSuccess) return hip_fail(e, "workspace zero kernel");
    ws_note_zeroed(ws, ws_bytes);
    return SEKV_OK;
}

sekv_status sekv_workspace_status(void *ws, size_t ws_bytes, hipStream_t stream,
                                  int32_t *error_bits) {
    if (!ws || !error_bits) return fail(SEKV_ERR_INVALID_ARG, "NULL argument");
    if (ws_bytes < sizeof(sekv::WsHeader)) return fail(SEKV_ERR_WORKSPACE, "workspace too small");
    sekv::WsHeader *h = static_cast<sekv::WsHeader *>(ws);
    int32_t v = 0;
    hipError_t e = hipMemcpyAsync(&v, &h->error, sizeof(v), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "reading the workspace error word");
    *error_bits = v;
    if (v) {
        const int32_t zero = 0;
        e = hipMemcpyAsync(&h->error, &zero, sizeof(zero), hipMemcpyHostToDevice, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) return hip_fail(e, "clearing the workspace error word");
    }
    return SEKV_OK;
}

sekv_status sekv_route_topk(const sekv_dims *dims, const sekv_cache *cache, int32_t *sel,
                            float *logits, void *ws, size_t ws_bytes, hipStream_t stream) {
    return run(sekv::kModeRoute, dims, cache, sel, logits, nullptr, nullptr, nullptr, ws,
               ws_bytes, stream);
}

sekv_status sekv_zoom_attend(const sekv_dims *dims, const sekv_cache *cache, const int32_t *sel,
                             const float *logits, void *out, void *ws, size_t ws_bytes,
                             hipStream_t stream) {
    return run(sekv::kModeAttend, dims, cache, nullptr, nullptr, sel, logits, out, ws, ws_bytes,
               stream);
}

sekv_status sekv_decode_step(const sekv_dims *dims, const sekv_cache *cache, int32_t *sel,
                             void *out, void *ws, size_t ws_bytes, hipStream_t stream) {
    return run(sekv::kModeFused, dims, cache, sel, nullptr, nullptr, nullptr, out, ws, ws_bytes,
               stream);
}

}  // extern "C"

namespace {

// Validate a learned-routing call and fill its launch parameters.  *launch is false when
// there is nothing to compute.
sekv_status gate_prepare(const sekv_dims *d, const sekv_cache *c, const sekv_gate *gt, int32_t *sel,
                         double *gate_logits, void *ws, size_t ws_bytes, sekv::GateParams *gp,
                         bool *launch) {
    *launch = false;
    sekv_status st = check_dims_impl(d);
    if (st != SEKV_OK) return st;
    st = check_cache(d, c, false);
    if (st != SEKV_OK) return st;
    st = check_ws(d, ws, ws_bytes);
    if (st != SEKV_OK) return st;
    if (!gt) return fail(SEKV_ERR_INVALID_ARG, "gate is NULL");
    const int dr = gt->route_dim;
    if (dr < 8 || dr > sekv::kGateMaxDr || dr % 8)
        return fail(SEKV_ERR_UNSUPPORTED, "route_dim %d: need a multiple of 8 in [8, %d]", dr,
                    sekv::kGateMaxDr);
    if (gt->reserved != 0) return fail(SEKV_ERR_INVALID_ARG, "gate.reserved must be 0");
    if (gt->budget_tokens < 0) return fail(SEKV_ERR_INVALID_ARG, "budget_tokens < 0");
    auto mis = [](const void *q, uintptr_t a) { return (reinterpret_cast<uintptr_t>(q) & (a - 1)) != 0; };
    if (!gt->proj || !gt->sum_route || !gt->thresholds)
        return fail(SEKV_ERR_INVALID_ARG, "gate proj, sum_route or thresholds is NULL");
    if (mis(gt->proj, 16) || mis(gt->sum_route, 16) || mis(gt->thresholds, 8) || mis(gate_logits, 8) ||
        mis(sel, 4))
        return fail(SEKV_ERR_INVALID_ARG, "gate arrays misaligned");
    if (d->batch == 0) return SEKV_OK;
    if (d->top_k > 0 && !sel) return fail(SEKV_ERR_INVALID_ARG, "sel is NULL");
    const sekv::Shape s = sekv::make_shape(*d);
    if (s.G > sekv::kGateMaxG || s.d > 128 || s.g_nrc * (s.k > 0 ? s.k : 1) > sekv::kGateMaxCand)
        return fail(SEKV_ERR_UNSUPPORTED, "shapes outside the learned-routing kernel's limits");
    const sekv::WsLayout L = sekv::make_layout(s);
    unsigned char *w = static_cast<unsigned char *>(ws);
    sekv::GateParams g{};
    g.B = s.B; g.Hq = s.Hq; g.Hkv = s.Hkv; g.G = s.G; g.d = s.d; g.dr = dr; g.k = s.k;
    g.M_max = s.M_max; g.cr = s.g_cr; g.n_rc = s.g_nrc;
    g.budget = gt->budget_tokens;
    g.scale_r = 1.0 / std::sqrt(double(dr));
    g.q = c->q; g.proj = gt->proj; g.sum_route = gt->sum_route;
    g.n_spans = c->n_spans; g.span_len = c->span_len; g.span_logsize = c->span_logsize;
    g.thr = gt->thresholds;
    g.sel = sel; g.gate_out = gate_logits;
    g.cnt = reinterpret_cast<uint32_t *>(w + L.gate_cnt);
    g.cand = reinterpret_cast<uint64_t *>(w + L.gate_cand);
    *gp = g;
    *launch = s.k > 0 || gate_logits != nullptr;
    return SEKV_OK;
}

sekv_status run_gate(const sekv_dims *d, const sekv_cache *c, const sekv_gate *gt, int32_t *sel,
                     double *gate_logits, void *ws, size_t ws_bytes, hipStream_t stream) {
    sekv::GateParams g{};
    bool launch = false;
    const sekv_status st = gate_prepare(d, c, gt, sel, gate_logits, ws, ws_bytes, &g, &launch);
    if (st != SEKV_OK || !launch) return st;
    hipError_t e = ws_prepare(ws, ws_bytes, sekv::layout_key(sekv::make_shape(*d)), 1, stream);
    if (e != hipSuccess) return hip_fail(e, "workspace zero kernel");
    e = sekv::launch_gate(g, d->dtype, stream);
    if (e != hipSuccess) return hip_fail(e, "learned-routing kernel launch");
    return SEKV_OK;
}

}  // namespace

extern "C" {

sekv_status sekv_route_gated(const sekv_dims *dims, const sekv_cache *cache, const sekv_gate *gate,
                             int32_t *sel, double *gate_logits, void *ws, size_t ws_bytes,
                             hipStream_t stream) {
    return run_gate(dims, cache, gate, sel, gate_logits, ws, ws_bytes, stream);
}

sekv_status sekv_decode_step_gated(const sekv_dims *dims, const sekv_cache *cache,
                                   const sekv_gate *gate, int32_t *sel, void *out, void *ws,
                                   size_t ws_bytes, hipStream_t stream) {
    // validate both halves before enqueuing either
    sekv::GateParams g{};
    bool launch = false;
    sekv_status st = gate_prepare(dims, cache, gate, sel, nullptr, ws, ws_bytes, &g, &launch);
    if (st != SEKV_OK) return st;
    sekv::Params p{};
    bool launch2 = false;
    st = prepare(sekv::kModeAttend, dims, cache, nullptr, nullptr, sel, nullptr, out, ws, ws_bytes, &p,
                 &launch2);
    if (st != SEKV_OK) return st;
    st = run_gate(dims, cache, gate, sel, nullptr, ws, ws_bytes, stream);
    if (st != SEKV_OK) return st;
    return run(sekv::kModeAttend, dims, cache, nullptr, nullptr, sel, nullptr, out, ws, ws_bytes, stream);
}

struct sekv_graph {
    hipGraph_t graph;
    hipGraphExec_t exec;
    int32_t n_layers;
    void *ws;
    size_t ws_bytes;
    uint64_t key;
};

sekv_status sekv_graph_create(const sekv_dims *dims, const sekv_cache *layers, int32_t n_layers,
                              int32_t *sel, void *out, void *ws, size_t ws_bytes,
                              sekv_graph **graph) {
    if (!graph) return fail(SEKV_ERR_INVALID_ARG, "graph is NULL");
    *graph = nullptr;
    if (n_layers < 1) return fail(SEKV_ERR_INVALID_ARG, "n_layers < 1");
    if (!layers) return fail(SEKV_ERR_INVALID_ARG, "layers is NULL");
    sekv_status st = check_dims_impl(dims);
    if (st != SEKV_OK) return st;
    // every layer is validated before anything is captured
    const size_t sel_stride = size_t(dims->batch) * dims->n_kv_heads * size_t(dims->top_k);
    const size_t out_stride = size_t(dims->batch) * dims->n_q_heads * size_t(dims->head_dim) *
                              (dims->out_dtype == SEKV_F32 ? 4 : 2);
    std::vector<sekv::Params> ps(static_cast<size_t>(n_layers));
    std::vector<char> go(static_cast<size_t>(n_layers));
    for (int32_t l = 0; l < n_layers; ++l) {
        bool launch = false;
        int32_t *sel_l = sel ? sel + size_t(l) * sel_stride : nullptr;
        void *out_l = out ? static_cast<unsigned char *>(out) + size_t(l) * out_stride : nullptr;
        st = prepare(sekv::kModeFused, dims, &layers[l], sel_l, nullptr, nullptr, nullptr, out_l,
                     ws, ws_bytes, &ps[size_t(l)], &launch);
        if (st != SEKV_OK) {
            char msg[512];
            std::snprintf(msg, sizeof(msg), "%s", sekv::last_error());
            return fail(st, "layer %d: %s", int(l), msg);
        }
        go[size_t(l)] = launch;
    }
    const int G = dims->n_q_heads / dims->n_kv_heads;
    // capture on a private stream (the legacy default stream cannot be captured); the
    // launches form one chain, so the layers share the workspace in order
    hipStream_t cs = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
    if (e != hipSuccess) return hip_fail(e, "capture stream");
    e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
        (void)hipStreamDestroy(cs);
        return hip_fail(e, "begin capture");
    }
    hipError_t le = hipSuccess;
    for (int32_t l = 0; l < n_layers && le == hipSuccess; ++l)
        if (go[size_t(l)]) le = sekv::launch_step(ps[size_t(l)], dims->dtype, dims->head_dim, G, cs);
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(cs, &g);
    (void)hipStreamDestroy(cs);
    if (le != hipSuccess || e != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        return hip_fail(le != hipSuccess ? le : e, "capturing the layer launches");
    }
    hipGraphExec_t x = nullptr;
    e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        (void)hipGraphDestroy(g);
        return hip_fail(e, "instantiating the graph");
    }
    sekv_graph *h = new (std::nothrow) sekv_graph{g, x, n_layers, ws, ws_bytes,
                                                  sekv::layout_key(sekv::make_shape(*dims))};
    if (!h) {
        (void)hipGraphExecDestroy(x);
        (void)hipGraphDestroy(g);
        return fail(SEKV_ERR_INVALID_ARG, "out of host memory");
    }
    *graph = h;
    return SEKV_OK;
}

sekv_status sekv_graph_launch(sekv_graph *graph, hipStream_t stream) {
    if (!graph) return fail(SEKV_ERR_INVALID_ARG, "graph is NULL");
    hipError_t e = ws_prepare(graph->ws, graph->ws_bytes, graph->key, uint64_t(graph->n_layers), stream);
    if (e != hipSuccess) return hip_fail(e, "workspace zero kernel");
    e = hipGraphLaunch(graph->exec, stream);
    if (e != hipSuccess) return hip_fail(e, "graph launch");
    return SEKV_OK;
}

sekv_status sekv_graph_destroy(sekv_graph *graph) {
    if (!graph) return SEKV_OK;
    hipError_t e = hipGraphExecDestroy(graph->exec);
    const hipError_t e2 = hipGraphDestroy(graph->graph);
    delete graph;
    if (e == hipSuccess) e = e2;
    if (e != hipSuccess) return hip_fail(e, "destroying the graph");
    return SEKV_OK;
}


// ------------------------------------------------------------------------------------
// pinned-host tier
// ------------------------------------------------------------------------------------
struct sekv_tier {
    sekv_dims dims;
    int32_t mode;               // SEKV_TIER_*
    int device;
    size_t slot_bytes;          // staging bytes per selection slot (largest block, aligned)
    size_t staging_bytes;
    int32_t *h_sel;             // pinned [B][Hkv][k]: selection read back per sequence (memcpy mode)
    int64_t *h_off;             // pinned [B][Hkv][M_max]: staging offsets (memcpy mode)
    void *d_mem;                // one device allocation: offsets | logits | stats | staging
    int64_t *d_off;             // [B][Hkv][M_max]
    float *d_logits;            // [B][Hq][M_max]
    unsigned long long *d_stats;  // [2]: bytes and blocks of the last step (gather mode)
    unsigned char *d_staging;   // [B][Hkv][k] slots
    hipEvent_t *ev_sel;         // [B] selection of sequence b is done (on main)
    hipEvent_t *ev_copy;        // [B] factors of sequence b are in staging (on side)
    hipEvent_t ev_t0, ev_t1;    // timing of the last step's copies (side stream)
    sekv::TierPlan plan;        // host plan of one sequence (memcpy mode)
    int64_t last_bytes;
    int32_t last_copies;
    bool timed;
    // layered steps (sekv_decode_layers_tiered), allocated on first use: two layer buffers,
    // each staging (prefetch region | miss region), staging offsets and prefetch records
    void *d_layer;
    unsigned char *d_lstage[2];
    int64_t *d_loff[2];
    int32_t *d_lpf[2];
    unsigned long long *d_lstats;  // [4]
    hipEvent_t ev_lsel, ev_lcopy;
};

sekv_status sekv_tier_create(const sekv_dims *dims, int32_t copy_mode, sekv_tier **tier) {
    if (!tier) return fail(SEKV_ERR_INVALID_ARG, "tier is NULL");
    *tier = nullptr;
    sekv_status st = check_dims_impl(dims);
    if (st != SEKV_OK) return st;
    if (dims->batch < 1) return fail(SEKV_ERR_INVALID_ARG, "the tier needs batch >= 1");
    if (copy_mode != SEKV_TIER_GATHER && copy_mode != SEKV_TIER_MEMCPY)
        return fail(SEKV_ERR_UNSUPPORTED, "tier copy mode %d", int(copy_mode));
    sekv_tier *t = new (std::nothrow) sekv_tier{};
    if (!t) return fail(SEKV_ERR_INVALID_ARG, "out of host memory");
    t->dims = *dims;
    t->mode = copy_mode;
    const size_t B = size_t(dims->batch), Hkv = size_t(dims->n_kv_heads), Hq = size_t(dims->n_q_heads);
    const size_t M = size_t(dims->max_spans), k = size_t(std::max(dims->top_k, 1));
    t->slot_bytes = sekv::align256(sekv::block_bytes(*dims, dims->max_span_len));
    t->staging_bytes = B * Hkv * k * t->slot_bytes;
    auto cleanup = [&](hipError_t e, const char *what) {
        sekv_tier_destroy(t);
        return hip_fail(e, what);
    };
    hipError_t e = hipGetDevice(&t->device);
    if (e != hipSuccess) return cleanup(e, "hipGetDevice");
    e = hipHostMalloc(reinterpret_cast<void **>(&t->h_sel), B * Hkv * k * sizeof(int32_t), hipHostMallocDefault);
    if (e != hipSuccess) return cleanup(e, "pinned selection mirror");
    e = hipHostMalloc(reinterpret_cast<void **>(&t->h_off), B * Hkv * M * sizeof(int64_t), hipHostMallocDefault);
    if (e != hipSuccess) return cleanup(e, "pinned offset table");
    std::memset(t->h_off, 0, B * Hkv * M * sizeof(int64_t));
    const size_t off_bytes = sekv::align256(B * Hkv * M * sizeof(int64_t));
    const size_t lg_bytes = sekv::align256(B * Hq * M * sizeof(float));
    e = hipMalloc(&t->d_mem, off_bytes + lg_bytes + 256 + t->staging_bytes);
    if (e != hipSuccess) return cleanup(e, "device staging");
    unsigned char *m = static_cast<unsigned char *>(t->d_mem);
    t->d_off = reinterpret_cast<int64_t *>(m);
    t->d_logits = reinterpret_cast<float *>(m + off_bytes);
    t->d_stats = reinterpret_cast<unsigned long long *>(m + off_bytes + lg_bytes);
    t->d_staging = m + off_bytes + lg_bytes + 256;
    e = hipMemset(t->d_mem, 0, off_bytes + lg_bytes + 256);
    if (e != hipSuccess) return cleanup(e, "clearing the offset table");
    t->ev_sel = new (std::nothrow) hipEvent_t[B]();
    t->ev_copy = new (std::nothrow) hipEvent_t[B]();
    if (!t->ev_sel || !t->ev_copy) {
        sekv_tier_destroy(t);
        return fail(SEKV_ERR_INVALID_ARG, "out of host memory");
    }
    for (size_t b = 0; b < B; ++b) {
        e = hipEventCreateWithFlags(&t->ev_sel[b], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&t->ev_copy[b], hipEventDisableTiming);
        if (e != hipSuccess) return cleanup(e, "creating events");
    }
    e = hipEventCreate(&t->ev_t0);
    if (e == hipSuccess) e = hipEventCreate(&t->ev_t1);
    if (e != hipSuccess) return cleanup(e, "creating timing events");
    *tier = t;
    return SEKV_OK;
}

sekv_status sekv_tier_destroy(sekv_tier *t) {
    if (!t) return SEKV_OK;
    const size_t B = size_t(std::max(t->dims.batch, 0));
    for (size_t b = 0; b < B; ++b) {
        if (t->ev_sel && t->ev_sel[b]) (void)hipEventDestroy(t->ev_sel[b]);
        if (t->ev_copy && t->ev_copy[b]) (void)hipEventDestroy(t->ev_copy[b]);
    }
    delete[] t->ev_sel;
    delete[] t->ev_copy;
    if (t->ev_t0) (void)hipEventDestroy(t->ev_t0);
    if (t->ev_t1) (void)hipEventDestroy(t->ev_t1);
    if (t->d_mem) (void)hipFree(t->d_mem);
    if (t->d_layer) (void)hipFree(t->d_layer);
    if (t->ev_lsel) (void)hipEventDestroy(t->ev_lsel);
    if (t->ev_lcopy) (void)hipEventDestroy(t->ev_lcopy);
    if (t->h_sel) (void)hipHostFree(t->h_sel);
    if (t->h_off) (void)hipHostFree(t->h_off);
    delete t;
    return SEKV_OK;
}

size_t sekv_tier_staging_size(const sekv_tier *t) { return t ? t->staging_bytes : 0; }

sekv_status sekv_tier_last_copy(sekv_tier *t, int64_t *bytes, int32_t *copies, float *ms) {
    if (!t || !bytes || !copies || !ms) return fail(SEKV_ERR_INVALID_ARG, "NULL argument");
    *ms = 0.0f;
    if (t->mode == SEKV_TIER_GATHER) {
        // the device counted them; valid once the step has completed
        unsigned long long st[2] = {0, 0};
        hipError_t e = hipMemcpy(st, t->d_stats, sizeof(st), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "reading the copy counters");
        t->last_bytes = int64_t(st[0]);
        t->last_copies = int32_t(st[1]);
    }
    *bytes = t->last_bytes;
    *copies = t->last_copies;
    if (t->timed) {
        const hipError_t e = hipEventElapsedTime(ms, t->ev_t0, t->ev_t1);
        if (e != hipSuccess) return hip_fail(e, "copy timing events");
    }
    return SEKV_OK;
}

sekv_status sekv_decode_step_tiered(const sekv_dims *dims, const sekv_cache *cache,
                                    const sekv_host_factors *host, sekv_tier *t, int32_t *sel,
                                    void *out, void *ws, size_t ws_bytes, hipStream_t main,
                                    hipStream_t side) {
    if (!t) return fail(SEKV_ERR_INVALID_ARG, "tier is NULL");
    sekv_status st = check_dims_impl(dims);
    if (st != SEKV_OK) return st;
    if (std::memcmp(dims, &t->dims, sizeof(sekv_dims)) != 0)
        return fail(SEKV_ERR_INVALID_ARG, "dims differ from the tier's");
    if (!cache || !host || !host->arena || !host->block_off || !host->span_len)
        return fail(SEKV_ERR_INVALID_ARG, "cache/host factor tables are NULL");
    if (host->arena_bytes <= 0) return fail(SEKV_ERR_INVALID_ARG, "arena_bytes <= 0");
    if ((host->block_rank == nullptr) != (cache->block_rank == nullptr))
        return fail(SEKV_ERR_INVALID_ARG, "host and device rank tables: both or neither");
    if (!out || (dims->top_k > 0 && !sel)) return fail(SEKV_ERR_INVALID_ARG, "sel/out is NULL");
    const bool gather = t->mode == SEKV_TIER_GATHER;
    if (gather && dims->top_k > 0 && (!cache->block_off || (reinterpret_cast<uintptr_t>(cache->block_off) & 7)))
        return fail(SEKV_ERR_INVALID_ARG, "gather mode needs cache.block_off: a device copy of the arena offsets");
    hipPointerAttribute_t attr{};
    if (hipPointerGetAttributes(&attr, host->arena) != hipSuccess || attr.type != hipMemoryTypeHost ||
        (gather && !attr.devicePointer)) {
        (void)hipGetLastError();
        return fail(SEKV_ERR_INVALID_ARG, "the host factor arena is not pinned%s memory",
                    gather ? ", device-mapped" : "");
    }
    const unsigned char *arena_dev = static_cast<const unsigned char *>(attr.devicePointer);
    const unsigned char *arena_host = static_cast<const unsigned char *>(host->arena);
    const int B = dims->batch, Hkv = dims->n_kv_heads, Hq = dims->n_q_heads, k = dims->top_k;
    const int M = dims->max_spans, d = dims->head_dim;
    const size_t oe = dims->out_dtype == SEKV_F32 ? 4 : 2;
    const size_t e = size_t(sekv::elem_bytes(dims->dtype));
    const int64_t region = int64_t(size_t(Hkv) * size_t(std::max(k, 1)) * t->slot_bytes);
    sekv_dims d1 = *dims;
    d1.batch = 1;
    // per-sequence views of the device cache (b is the outermost index of every array)
    auto seq_cache = [&](int b) {
        sekv_cache c = *cache;
        const size_t bb = size_t(b);
        c.q = static_cast<const unsigned char *>(cache->q) + bb * Hq * d * e;
        c.anchor_k = cache->anchor_k ? static_cast<const unsigned char *>(cache->anchor_k) +
                                           bb * Hkv * size_t(dims->max_anchors) * d * e : nullptr;
        c.anchor_v = cache->anchor_v ? static_cast<const unsigned char *>(cache->anchor_v) +
                                           bb * Hkv * size_t(dims->max_anchors) * d * e : nullptr;
        c.n_anchors = cache->n_anchors + bb;
        c.sum_k = static_cast<const unsigned char *>(cache->sum_k) + bb * Hkv * size_t(M) * d * e;
        c.sum_v = static_cast<const unsigned char *>(cache->sum_v) + bb * Hkv * size_t(M) * d * e;
        c.n_spans = cache->n_spans + bb;
        c.span_len = cache->span_len + bb * M;
        c.span_logsize = cache->span_logsize + bb * M;
        c.factors = t->d_staging;
        c.factors_bytes = int64_t(t->staging_bytes);
        c.block_off = t->d_off + bb * Hkv * M;
        c.block_rank = cache->block_rank ? cache->block_rank + bb * Hkv * M : nullptr;
        return c;
    };
    hipError_t he = hipSuccess;
    t->timed = false;
    // 1. routing per sequence on the main stream
    for (int b = 0; b < B; ++b) {
        sekv_cache c = seq_cache(b);
        st = run(sekv::kModeRoute, &d1, &c, sel ? sel + size_t(b) * Hkv * k : nullptr,
                 t->d_logits + size_t(b) * Hq * M, nullptr, nullptr, nullptr, ws, ws_bytes, main);
        if (st != SEKV_OK) return st;
        if (k > 0) {
            if (!gather)
                he = hipMemcpyAsync(t->h_sel + size_t(b) * Hkv * k, sel + size_t(b) * Hkv * k,
                                    size_t(Hkv) * k * sizeof(int32_t), hipMemcpyDeviceToHost, main);
            if (he == hipSuccess) he = hipEventRecord(t->ev_sel[b], main);
            if (he != hipSuccess) return hip_fail(he, "selection readback");
        }
    }
    // 2. per sequence: its selected blocks go to staging on the side stream (overlapping
    //    the routing of later sequences), then its attention runs on the main stream
    int64_t bytes = 0;
    int32_t copies = 0;
    bool first = true;
    for (int b = 0; b < B; ++b) {
        if (k > 0 && gather) {
            he = hipStreamWaitEvent(side, t->ev_sel[b], 0);
            if (b == 0) {
                // the copy time runs from the first sequence's selection
                if (he == hipSuccess) he = hipEventRecord(t->ev_t0, side);
                if (he == hipSuccess) he = sekv::launch_stats_reset(t->d_stats, side);
            }
            sekv::TierGatherArgs a{};
            a.arena = arena_dev;
            a.staging = t->d_staging;
            a.sel = sel + size_t(b) * Hkv * k;
            a.span_len = cache->span_len + size_t(b) * M;
            a.block_off = cache->block_off + size_t(b) * Hkv * M;
            a.block_rank = cache->block_rank ? cache->block_rank + size_t(b) * Hkv * M : nullptr;
            a.stage_off = t->d_off + size_t(b) * Hkv * M;
            a.stats = t->d_stats;
            a.error = &static_cast<sekv::WsHeader *>(ws)->error;
            a.arena_bytes = host->arena_bytes;
            a.slot0 = int64_t(b) * region;
            a.slot_bytes = int64_t(t->slot_bytes);
            a.Hkv = Hkv; a.k = k; a.M = M; a.r = dims->rank; a.d = d; a.elem = int32_t(e);
            a.max_span_len = dims->max_span_len;
            a.chunks_per_slot = int32_t((t->slot_bytes + sekv::kGatherChunk - 1) / sekv::kGatherChunk);
            if (he == hipSuccess) he = sekv::launch_tier_gather(a, side);
            // the timing event before the last join, so a capture of the step ends joined
            if (he == hipSuccess && b == B - 1) he = hipEventRecord(t->ev_t1, side);
            if (he == hipSuccess) he = hipEventRecord(t->ev_copy[b], side);
            if (he == hipSuccess) he = hipStreamWaitEvent(main, t->ev_copy[b], 0);
            if (he != hipSuccess) return hip_fail(he, "factor gather");
        } else if (k > 0) {
            he = hipEventSynchronize(t->ev_sel[b]);
            if (he != hipSuccess) return hip_fail(he, "waiting for the selection");
            sekv::TierPlanIn in{dims, b, t->h_sel + size_t(b) * Hkv * k, host->span_len + size_t(b) * M,
                                host->block_off + size_t(b) * Hkv * M, host->arena_bytes,
                                int64_t(b) * region, region,
                                host->block_rank ? host->block_rank + size_t(b) * Hkv * M : nullptr};
            st = sekv::plan_tier_sequence(in, &t->plan);
            if (st != SEKV_OK) return st;
            int64_t *hoff = t->h_off + size_t(b) * Hkv * M;
            for (int32_t i : t->plan.off_set) hoff[i] = t->plan.off[size_t(i)];
            if (first && !t->plan.runs.empty()) {
                he = hipEventRecord(t->ev_t0, side);
                if (he != hipSuccess) return hip_fail(he, "copy timing event");
                first = false;
            }
            for (const sekv::TierRun &r : t->plan.runs) {
                he = hipMemcpyAsync(t->d_staging + r.dst, arena_host + r.src, size_t(r.bytes),
                                    hipMemcpyHostToDevice, side);
                if (he != hipSuccess) return hip_fail(he, "factor copy");
            }
            bytes += t->plan.bytes;
            copies += int32_t(t->plan.runs.size());
            he = hipMemcpyAsync(t->d_off + size_t(b) * Hkv * M, hoff, size_t(Hkv) * M * sizeof(int64_t),
                                hipMemcpyHostToDevice, side);
            if (he == hipSuccess) he = hipEventRecord(t->ev_copy[b], side);
            if (he == hipSuccess) he = hipStreamWaitEvent(main, t->ev_copy[b], 0);
            if (he != hipSuccess) return hip_fail(he, "staging offsets");
        }
        sekv_cache c = seq_cache(b);
        st = run(sekv::kModeAttend, &d1, &c, nullptr, nullptr, sel ? sel + size_t(b) * Hkv * k : nullptr,
                 t->d_logits + size_t(b) * Hq * M, static_cast<unsigned char *>(out) + size_t(b) * Hq * d * oe,
                 ws, ws_bytes, main);
        if (st != SEKV_OK) return st;
    }
    if (gather && k > 0) {
        t->timed = true;
    } else if (!first) {
        he = hipEventRecord(t->ev_t1, side);
        if (he != hipSuccess) return hip_fail(he, "copy timing event");
        t->timed = true;
    }
    if (!gather) {
        t->last_bytes = bytes;
        t->last_copies = copies;
    }
    return SEKV_OK;
}

sekv_status sekv_decode_layers_tiered(const sekv_dims *dims, const sekv_cache *caches,
                                      const sekv_host_factors *hosts, int32_t n_layers, int32_t prefetch,
                                      sekv_tier *t, int32_t *sel, void *out, void *ws, size_t ws_bytes,
                                      hipStream_t main, hipStream_t side) {
    if (!t) return fail(SEKV_ERR_INVALID_ARG, "tier is NULL");
    sekv_status st = check_dims_impl(dims);
    if (st != SEKV_OK) return st;
    if (std::memcmp(dims, &t->dims, sizeof(sekv_dims)) != 0)
        return fail(SEKV_ERR_INVALID_ARG, "dims differ from the tier's");
    if (t->mode != SEKV_TIER_GATHER) return fail(SEKV_ERR_UNSUPPORTED, "layered steps need a gather-mode tier");
    if (n_layers < 1 || !caches || !hosts) return fail(SEKV_ERR_INVALID_ARG, "n_layers < 1 or NULL layer arrays");
    if (prefetch != 0 && prefetch != 1) return fail(SEKV_ERR_INVALID_ARG, "prefetch must be 0 or 1");
    const int B = dims->batch, Hkv = dims->n_kv_heads, Hq = dims->n_q_heads, k = dims->top_k;
    const int M = dims->max_spans, d = dims->head_dim;
    if (!out || (k > 0 && !sel)) return fail(SEKV_ERR_INVALID_ARG, "sel/out is NULL");
    const size_t oe = dims->out_dtype == SEKV_F32 ? 4 : 2;
    const size_t e = size_t(sekv::elem_bytes(dims->dtype));
    std::vector<const unsigned char *> arena_dev(size_t(n_layers), nullptr);
    for (int l = 0; l < n_layers; ++l) {
        const sekv_cache &c = caches[l];
        const sekv_host_factors &h = hosts[l];
        if (!h.arena || !h.block_off || !h.span_len || h.arena_bytes <= 0)
            return fail(SEKV_ERR_INVALID_ARG, "layer %d: host factor tables are NULL or empty", l);
        if ((h.block_rank == nullptr) != (c.block_rank == nullptr))
            return fail(SEKV_ERR_INVALID_ARG, "layer %d: host and device rank tables: both or neither", l);
        if (k > 0 && (!c.block_off || (reinterpret_cast<uintptr_t>(c.block_off) & 7)))
            return fail(SEKV_ERR_INVALID_ARG, "layer %d: cache.block_off must be a device copy of the arena offsets", l);
        hipPointerAttribute_t attr{};
        if (hipPointerGetAttributes(&attr, h.arena) != hipSuccess || attr.type != hipMemoryTypeHost ||
            !attr.devicePointer) {
            (void)hipGetLastError();
            return fail(SEKV_ERR_INVALID_ARG, "layer %d: the host factor arena is not pinned, device-mapped memory", l);
        }
        arena_dev[size_t(l)] = static_cast<const unsigned char *>(attr.devicePointer);
    }
    const size_t slots = size_t(B) * Hkv * size_t(std::max(k, 1));
    const size_t region = slots * t->slot_bytes;
    hipError_t he = hipSuccess;
    if (!t->d_layer) {
        // two layer buffers: staging (prefetch | miss), offsets, prefetch records; counters
        const size_t off_b = sekv::align256(size_t(B) * Hkv * M * sizeof(int64_t));
        const size_t pf_b = sekv::align256(slots * sizeof(int32_t));
        const size_t per = 2 * region + off_b + pf_b;
        he = hipMalloc(&t->d_layer, 2 * per + 256);
        if (he != hipSuccess) return hip_fail(he, "layered staging");
        unsigned char *m = static_cast<unsigned char *>(t->d_layer);
        for (int i = 0; i < 2; ++i) {
            unsigned char *base = m + size_t(i) * per;
            t->d_lstage[i] = base;
            t->d_loff[i] = reinterpret_cast<int64_t *>(base + 2 * region);
            t->d_lpf[i] = reinterpret_cast<int32_t *>(base + 2 * region + off_b);
        }
        t->d_lstats = reinterpret_cast<unsigned long long *>(m + 2 * per);
        he = hipMemset(t->d_layer, 0, 2 * per + 256);
        if (he == hipSuccess) he = hipEventCreateWithFlags(&t->ev_lsel, hipEventDisableTiming);
        if (he == hipSuccess) he = hipEventCreateWithFlags(&t->ev_lcopy, hipEventDisableTiming);
        if (he != hipSuccess) {
            if (t->ev_lsel) (void)hipEventDestroy(t->ev_lsel);
            (void)hipFree(t->d_layer);
            t->d_layer = nullptr;
            t->ev_lsel = nullptr;
            return hip_fail(he, "layered staging set-up");
        }
    }
    const int chunks = int32_t((t->slot_bytes + sekv::kGatherChunk - 1) / sekv::kGatherChunk);
    auto copy_args = [&](int l, int buf, const int32_t *which, int pf, int use_pf) {
        sekv::LayerCopyArgs a{};
        a.arena = arena_dev[size_t(l)];
        a.staging = t->d_lstage[buf];
        a.sel = which;
        a.span_len = caches[l].span_len;
        a.block_off = caches[l].block_off;
        a.block_rank = caches[l].block_rank;
        a.stage_off = t->d_loff[buf];
        a.pf_span = t->d_lpf[buf];
        a.stats = t->d_lstats;
        a.error = &static_cast<sekv::WsHeader *>(ws)->error;
        a.arena_bytes = hosts[l].arena_bytes;
        a.slot_bytes = int64_t(t->slot_bytes);
        a.miss0 = int64_t(region);
        a.B = B; a.Hkv = Hkv; a.k = k; a.M = M; a.r = dims->rank; a.d = d; a.elem = int32_t(e);
        a.max_span_len = dims->max_span_len; a.chunks_per_slot = chunks;
        a.prefetch = pf; a.use_pf = use_pf;
        return a;
    };
    he = sekv::launch_stats_reset4(t->d_lstats, side);
    if (he != hipSuccess) return hip_fail(he, "layer counters");
    for (int l = 0; l < n_layers; ++l) {
        const int buf = l & 1;
        int32_t *sel_l = k > 0 ? sel + size_t(l) * B * Hkv * k : nullptr;
        sekv_cache c = caches[l];
        c.factors = t->d_lstage[buf];
        c.factors_bytes = int64_t(2 * region);
        c.block_off = t->d_loff[buf];
        // 1. routing and selection of layer l (after layer l - 1's attention on main)
        st = run(sekv::kModeRoute, dims, &c, sel_l, t->d_logits, nullptr, nullptr, nullptr, ws, ws_bytes, main);
        if (st != SEKV_OK) return st;
        if (k > 0) {
            // 2. the blocks layer l selected that are not in its staging yet
            he = hipEventRecord(t->ev_lsel, main);
            if (he == hipSuccess) he = hipStreamWaitEvent(side, t->ev_lsel, 0);
            if (he == hipSuccess) he = sekv::launch_layer_copy(copy_args(l, buf, sel_l, 0, prefetch && l > 0), side);
            if (he == hipSuccess) he = hipEventRecord(t->ev_lcopy, side);
            // 3. layer l + 1's blocks of the spans layer l selected, behind layer l's attention
            if (he == hipSuccess && prefetch && l + 1 < n_layers)
                he = sekv::launch_layer_copy(copy_args(l + 1, buf ^ 1, sel_l, 1, 0), side);
            if (he == hipSuccess) he = hipStreamWaitEvent(main, t->ev_lcopy, 0);
            if (he != hipSuccess) return hip_fail(he, "layered copies");
        }
        // 4. layer l's attention from staging
        st = run(sekv::kModeAttend, dims, &c, nullptr, nullptr, sel_l, t->d_logits,
                 static_cast<unsigned char *>(out) + size_t(l) * B * Hq * d * oe, ws, ws_bytes, main);
        if (st != SEKV_OK) return st;
    }
    // the side stream's last work (a prefetch nobody uses is not enqueued) joins main
    he = hipEventRecord(t->ev_lcopy, side);
    if (he == hipSuccess) he = hipStreamWaitEvent(main, t->ev_lcopy, 0);
    if (he != hipSuccess) return hip_fail(he, "joining the copy stream");
    return SEKV_OK;
}

sekv_status sekv_tier_layer_stats(sekv_tier *t, int64_t stats[4]) {
    if (!t || !stats) return fail(SEKV_ERR_INVALID_ARG, "NULL argument");
    for (int i = 0; i < 4; ++i) stats[i] = 0;
    if (!t->d_layer) return SEKV_OK;
    unsigned long long st[4] = {0, 0, 0, 0};
    const hipError_t e = hipMemcpy(st, t->d_lstats, sizeof(st), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "reading the layer copy counters");
    for (int i = 0; i < 4; ++i) stats[i] = int64_t(st[i]);
    return SEKV_OK;
}

sekv_status sekv_validate_cache(const sekv_dims *dims, const sekv_cache *host_copy) {
    return sekv::validate_cache(dims, host_copy);
}

}  // extern "C"
