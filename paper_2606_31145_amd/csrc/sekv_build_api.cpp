// C ABI of the prefill-side builder: host checks, the arena layout, launches.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>

#include "sekv.h"
#include "sekv_host.h"
#include "sekv_internal.h"
#include "sekv_build_internal.h"

namespace {

using sekv::check_build_dims;
using sekv::fail;

bool misaligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; }

size_t seg_ws(const sekv_build_dims &d) {
    const size_t B = size_t(d.batch), N = size_t(d.max_tokens);
    auto a16 = [](size_t x) { return (x + 15) & ~size_t(15); };
    return a16(B * N) * 2 + a16(B * (N + 2) * 4);
}

}  // namespace

extern "C" {

size_t sekv_segment_workspace_size(const sekv_build_dims *dims) {
    if (check_build_dims(dims) != SEKV_OK) return 0;
    return seg_ws(*dims);
}

sekv_status sekv_segment(const sekv_build_dims *dims, const float *surprisal, const int32_t *n_tokens,
                         int32_t *n_anchors, int32_t *anchor_idx, int32_t *n_spans, int32_t *span_start,
                         int32_t *span_len, void *ws, size_t ws_bytes, hipStream_t stream) {
    sekv_status st = check_build_dims(dims);
    if (st != SEKV_OK) return st;
    if (dims->batch == 0) return SEKV_OK;
    if (!surprisal || !n_tokens || !n_anchors || !anchor_idx || !n_spans || !span_start || !span_len || !ws)
        return fail(SEKV_ERR_INVALID_ARG, "NULL argument");
    if (misaligned(surprisal, 4) || misaligned(n_tokens, 4) || misaligned(anchor_idx, 4) ||
        misaligned(span_start, 4) || misaligned(span_len, 4) || misaligned(ws, 16))
        return fail(SEKV_ERR_INVALID_ARG, "misaligned argument");
    if (ws_bytes < seg_ws(*dims)) return fail(SEKV_ERR_WORKSPACE, "segmentation workspace too small");
    const size_t B = size_t(dims->batch), N = size_t(dims->max_tokens);
    auto a16 = [](size_t x) { return (x + 15) & ~size_t(15); };
    unsigned char *w = static_cast<unsigned char *>(ws);
    sekv::SegArgs a{};
    a.surprisal = surprisal; a.n_tokens = n_tokens;
    a.n_anchors = n_anchors; a.anchor_idx = anchor_idx;
    a.n_spans = n_spans; a.span_start = span_start; a.span_len = span_len;
    a.ws_flag = w;
    a.ws_inspan = w + a16(B * N);
    a.ws_pos = reinterpret_cast<int32_t *>(w + 2 * a16(B * N));
    a.alpha = dims->alpha;
    a.N = dims->max_tokens; a.min_span = dims->min_span; a.window = dims->window;
    const hipError_t e = sekv::launch_segment(a, dims->batch, stream);
    if (e != hipSuccess) return fail(SEKV_ERR_HIP, "segmentation launch: %s", hipGetErrorString(e));
    return SEKV_OK;
}

int64_t sekv_build_layout(const sekv_build_dims *dims, int32_t max_spans, const int32_t *n_spans,
                          const int32_t *span_len, int64_t *block_off, int32_t *block_rank) {
    return sekv::build_layout(dims, max_spans, n_spans, span_len, block_off, block_rank);
}

sekv_status sekv_build_cache(const sekv_build_dims *dims, const void *keys, const void *values,
                             const float *surprisal, const int32_t *n_tokens, const int32_t *n_anchors,
                             const int32_t *anchor_idx, const int32_t *n_spans, const int32_t *span_start,
                             const int32_t *span_len_seg, const float *omega, int32_t max_anchors,
                             int32_t max_spans, void *anchor_k, void *anchor_v, void *sum_k, void *sum_v,
                             int32_t *span_len, double *span_logsize, void *factors, int64_t factors_bytes,
                             const int64_t *block_off, void *ws, size_t ws_bytes, hipStream_t stream) {
    sekv_status st = check_build_dims(dims);
    if (st != SEKV_OK) return st;
    if (dims->batch == 0) return SEKV_OK;
    if (max_anchors < 1 || max_spans < 1) return fail(SEKV_ERR_INVALID_ARG, "max_anchors/max_spans < 1");
    const void *req[] = {keys, values, surprisal, n_tokens, n_anchors, anchor_idx, n_spans, span_start,
                         span_len_seg, omega, anchor_k, anchor_v, sum_k, sum_v, span_len, span_logsize,
                         factors, block_off, ws};
    for (const void *p : req)
        if (!p) return fail(SEKV_ERR_INVALID_ARG, "NULL argument");
    if (misaligned(keys, 16) || misaligned(values, 16) || misaligned(anchor_k, 16) || misaligned(anchor_v, 16) ||
        misaligned(sum_k, 16) || misaligned(sum_v, 16) || misaligned(factors, 16) || misaligned(block_off, 8) ||
        misaligned(span_logsize, 8) || misaligned(omega, 4) || misaligned(ws, 256))
        return fail(SEKV_ERR_INVALID_ARG, "misaligned argument");
    if (factors_bytes <= 0) return fail(SEKV_ERR_INVALID_ARG, "factors_bytes <= 0");
    if (ws_bytes < sizeof(sekv::WsHeader)) return fail(SEKV_ERR_WORKSPACE, "workspace too small");
    sekv::BuildArgs a{};
    a.keys = keys; a.values = values; a.surprisal = surprisal; a.n_tokens = n_tokens;
    a.n_anchors = n_anchors; a.anchor_idx = anchor_idx; a.n_spans = n_spans; a.span_start = span_start;
    a.span_len_seg = span_len_seg; a.omega = omega;
    a.anchor_k = anchor_k; a.anchor_v = anchor_v; a.sum_k = sum_k; a.sum_v = sum_v;
    a.span_len_out = span_len; a.span_logsize = span_logsize;
    a.factors = factors; a.factors_bytes = factors_bytes; a.block_off = block_off;
    a.error = &static_cast<sekv::WsHeader *>(ws)->error;
    a.Hkv = dims->n_kv_heads; a.N = dims->max_tokens; a.d = dims->head_dim;
    a.elem = sekv::elem_bytes(dims->dtype); a.R = dims->rank; a.l = dims->sketch; a.sweeps = dims->sweeps;
    a.power = dims->power;
    size_t tb = 0;
    a.trace = sekv::trace_buffer(&tb);
    a.trace_items = a.trace ? int64_t(tb / (sizeof(int64_t) * sekv::kTraceSlots)) : 0;
    a.A_max = max_anchors; a.M_max = max_spans;
    const hipError_t e = sekv::launch_build(a, dims->batch, stream);
    if (e != hipSuccess) return fail(SEKV_ERR_HIP, "builder launch: %s", hipGetErrorString(e));
    return SEKV_OK;
}

}  // extern "C"
