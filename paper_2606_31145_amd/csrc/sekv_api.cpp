// C ABI of the SeKV decode-step library: host-side validation, workspace layout and
// launch set-up.  Every check that can be made on the host is made here, before
// anything is enqueued; the kernels clamp device-side table values on their own.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "sekv.h"
#include "sekv_internal.h"

namespace {

thread_local char g_err[512] = "";

sekv_status fail(sekv_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

sekv_status hip_fail(hipError_t e, const char *what) {
    return fail(SEKV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

sekv_status check_dims_impl(const sekv_dims *d) {
    if (!d) return fail(SEKV_ERR_INVALID_ARG, "dims is NULL");
    if (d->batch < 0) return fail(SEKV_ERR_INVALID_ARG, "batch < 0");
    if (d->n_q_heads <= 0 || d->n_kv_heads <= 0)
        return fail(SEKV_ERR_INVALID_ARG, "head counts must be positive");
    if (d->n_q_heads % d->n_kv_heads)
        return fail(SEKV_ERR_INVALID_ARG, "n_q_heads %% n_kv_heads != 0");
    const int G = d->n_q_heads / d->n_kv_heads;
    if (G != 1 && G != 2 && G != 4 && G != 8)
        return fail(SEKV_ERR_UNSUPPORTED, "group size %d not in {1,2,4,8}", G);
    if (d->head_dim != 64 && d->head_dim != 128)
        return fail(SEKV_ERR_UNSUPPORTED, "head_dim %d not in {64,128}", d->head_dim);
    if (d->rank != 8 && d->rank != 16 && d->rank != 32 && d->rank != 64)
        return fail(SEKV_ERR_UNSUPPORTED, "rank %d: need 8, 16, 32 or 64", d->rank);
    if (d->top_k < 0 || d->top_k > sekv::kMaxTopK)
        return fail(SEKV_ERR_UNSUPPORTED, "top_k %d not in [0,%d]", d->top_k, sekv::kMaxTopK);
    if (d->max_anchors < 0) return fail(SEKV_ERR_INVALID_ARG, "max_anchors < 0");
    if (d->max_spans < 1) return fail(SEKV_ERR_INVALID_ARG, "max_spans < 1");
    if (d->max_span_len < 1) return fail(SEKV_ERR_INVALID_ARG, "max_span_len < 1");
    if (d->dtype != SEKV_F32 && d->dtype != SEKV_BF16)
        return fail(SEKV_ERR_UNSUPPORTED, "dtype %d", d->dtype);
    if (d->out_dtype != SEKV_F32 && d->out_dtype != SEKV_BF16)
        return fail(SEKV_ERR_UNSUPPORTED, "out_dtype %d", d->out_dtype);
    if (d->dtype == SEKV_F32 && d->out_dtype != SEKV_F32)
        return fail(SEKV_ERR_UNSUPPORTED, "float32 storage needs float32 output");
    const int zoom = d->flags & 3;
    if ((d->flags & ~3) || zoom > SEKV_ZOOM_FACTORED)
        return fail(SEKV_ERR_UNSUPPORTED, "flags 0x%x", unsigned(d->flags));
    if (!(d->softmax_scale > 0.0) || !std::isfinite(d->softmax_scale))
        return fail(SEKV_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
    if (d->max_spans > sekv::kMaxSpans)
        return fail(SEKV_ERR_UNSUPPORTED, "max_spans %d > %d", d->max_spans, sekv::kMaxSpans);
    const long long rows = (long long)d->batch * d->n_kv_heads * std::max(d->max_spans, d->max_anchors);
    if (rows > (1ll << 31)) return fail(SEKV_ERR_UNSUPPORTED, "tables too large");
    return SEKV_OK;
}

sekv_status check_cache(const sekv_dims *d, const sekv_cache *c, bool need_factors) {
    if (!c) return fail(SEKV_ERR_INVALID_ARG, "cache is NULL");
    if (d->batch == 0) return SEKV_OK;
    struct { const void *p; const char *name; } ptrs[] = {
        {c->q, "q"}, {c->sum_k, "sum_k"}, {c->sum_v, "sum_v"}, {c->n_spans, "n_spans"},
        {c->span_len, "span_len"}, {c->span_logsize, "span_logsize"},
        {c->n_anchors, "n_anchors"}};
    for (auto &x : ptrs) {
        if (!x.p) return fail(SEKV_ERR_INVALID_ARG, "cache.%s is NULL", x.name);
        if (!aligned16(x.p)) return fail(SEKV_ERR_INVALID_ARG, "cache.%s not 16-byte aligned", x.name);
    }
    if (d->max_anchors > 0) {
        if (!c->anchor_k || !c->anchor_v)
            return fail(SEKV_ERR_INVALID_ARG, "cache.anchor_k/anchor_v is NULL");
        if (!aligned16(c->anchor_k) || !aligned16(c->anchor_v))
            return fail(SEKV_ERR_INVALID_ARG, "anchor arrays not 16-byte aligned");
    }
    if (need_factors && d->top_k > 0) {
        if (!c->factors || !c->block_off)
            return fail(SEKV_ERR_INVALID_ARG, "cache.factors/block_off is NULL");
        if (!aligned16(c->factors) || !aligned16(c->block_off))
            return fail(SEKV_ERR_INVALID_ARG, "factor arena or offsets not 16-byte aligned");
        if (c->factors_bytes <= 0) return fail(SEKV_ERR_INVALID_ARG, "factors_bytes <= 0");
    }
    return SEKV_OK;
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
    if ((sel_out && !aligned16(sel_out)) || (sel_in && !aligned16(sel_in)) ||
        (out && !aligned16(out)) || (logits_out && !aligned16(logits_out)) ||
        (logits_in && !aligned16(logits_in)))
        return fail(SEKV_ERR_INVALID_ARG, "sel/logits/out not 16-byte aligned");

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
    p.sel_out = sel_out; p.logits_out = logits_out; p.sel_in = sel_in; p.logits_in = logits_in;
    p.out = out;
    p.hdr = reinterpret_cast<sekv::WsHeader *>(w);
    p.route_cnt = reinterpret_cast<uint32_t *>(w + L.route_cnt);
    p.sel_ready = reinterpret_cast<uint32_t *>(w + L.sel_ready);
    p.part_cnt = reinterpret_cast<uint32_t *>(w + L.part_cnt);
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
    *pp = p;
    *launch = p.end_share > 0;
    return SEKV_OK;
}

sekv_status run(int mode, const sekv_dims *d, const sekv_cache *c, int32_t *sel_out,
                float *logits_out, const int32_t *sel_in, const float *logits_in, void *out,
                void *ws, size_t ws_bytes, hipStream_t stream) {
    sekv::Params p{};
    bool launch = false;
    const sekv_status st = prepare(mode, d, c, sel_out, logits_out, sel_in, logits_in, out, ws,
                                   ws_bytes, &p, &launch);
    if (st != SEKV_OK || !launch) return st;
    const hipError_t e = sekv::launch_step(p, d->dtype, d->head_dim, d->n_q_heads / d->n_kv_heads,
                                           stream);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return SEKV_OK;
}

}  // namespace

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

const char *sekv_last_error(void) { return g_err; }

sekv_status sekv_check_dims(const sekv_dims *dims) { return check_dims_impl(dims); }

size_t sekv_workspace_size(const sekv_dims *dims) {
    char saved[sizeof(g_err)];
    std::memcpy(saved, g_err, sizeof(g_err));
    const sekv_status st = check_dims_impl(dims);
    std::memcpy(g_err, saved, sizeof(g_err));
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

struct sekv_graph {
    hipGraph_t graph;
    hipGraphExec_t exec;
    int32_t n_layers;
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
            char msg[sizeof(g_err)];
            std::snprintf(msg, sizeof(msg), "%s", g_err);
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
    sekv_graph *h = new (std::nothrow) sekv_graph{g, x, n_layers};
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
    const hipError_t e = hipGraphLaunch(graph->exec, stream);
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

}  // extern "C"
