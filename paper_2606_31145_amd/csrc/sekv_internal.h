// Internal definitions shared by the host layer (sekv_api.cpp) and the kernels
// (sekv_kernels.hip): launch parameters and the workspace layout.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>
#include <hip/hip_vector_types.h>

#include "sekv.h"

namespace sekv {

// Work decomposition (compile-time tile sizes).
constexpr int kThreads = 256;      // threads per workgroup: 4 wave64s
constexpr int kRouteChunk = 128;   // spans per routing / summary work item
// Anchor tokens per anchor work item: 8 key + 8 value vectors of 16 bytes per thread.
constexpr int anchor_chunk(int elem_bytes, int head_dim) { return 32768 / (head_dim * elem_bytes); }
constexpr int kZoomBlock = 512;    // tokens of a zoomed span scored per LDS pass
constexpr int kMaxTopK = 64;
constexpr int kMergeBuf = 512;     // candidates ranked in LDS
constexpr int kLoserWin = 128;     // losing candidates folded per window (single merger)
constexpr int kZoomLosers = 32;    // losing candidates folded by one zoom item, at most

enum Mode : int32_t { kModeRoute = 0, kModeAttend = 1, kModeFused = 2 };

// Device error bits (workspace header word `error`).
enum : int32_t { kErrSpinTimeout = 1, kErrBlockRange = 2, kErrSelRange = 4 };

// Workspace header: dynamic work counter and shutdown counter, then per-(b, kv head)
// counters.  The last workgroup to finish a launch zeroes every counter it used.
struct WsHeader {
    uint32_t ticket;
    uint32_t exit_count;
    int32_t error;
    uint32_t pad[61];
};

// Byte offsets of the workspace sections for one dims.
struct WsLayout {
    size_t route_cnt, sel_ready, part_cnt;    // uint32 [P]
    size_t zrec;                              // int32x4 [P][k]: span, |S|, offset lo/hi
    size_t cand_key;                          // uint64 [P][n_rc][kc]
    size_t cand_idx;                          // int32  [P][n_rc][kc]
    size_t cand_len;                          // int32  [P][n_rc][kc]  |S|
    size_t cand_off;                          // int64  [P][n_rc][kc]  block offset
    size_t cand_cnt;                          // int32  [P][n_rc]
    size_t cand_lg;                           // float  [P][n_rc][kc][G]
    size_t part_ml;                           // float  [P][n_slots][G][2]
    size_t part_o;                            // float  [P][n_slots][G][d]
    size_t total;
};

struct Shape {
    int B, Hq, Hkv, G, d, r, k, A_max, M_max, L_max;
    int P;        // B * Hkv pairs
    int n_rc;     // routing/summary chunks per pair
    int n_ac;     // anchor chunks per pair
    int kc;       // candidates kept per routing chunk = min(k, kRouteChunk)
    int n_slots;  // partials per pair (fused layout: anchors, summaries, losers, zoom)
};

inline int elem_bytes(int dtype) { return dtype == SEKV_BF16 ? 2 : 4; }

inline Shape make_shape(const sekv_dims &d) {
    Shape s{};
    s.B = d.batch; s.Hq = d.n_q_heads; s.Hkv = d.n_kv_heads; s.G = s.Hq / s.Hkv;
    s.d = d.head_dim; s.r = d.rank; s.k = d.top_k;
    s.A_max = d.max_anchors; s.M_max = d.max_spans; s.L_max = d.max_span_len;
    s.P = s.B * s.Hkv;
    s.n_rc = (s.M_max + kRouteChunk - 1) / kRouteChunk;
    const int ca = anchor_chunk(elem_bytes(d.dtype), s.d);
    s.n_ac = (s.A_max + ca - 1) / ca;
    s.kc = s.k < kRouteChunk ? s.k : kRouteChunk;
    s.n_slots = s.n_ac + s.n_rc + 1 + s.k;
    return s;
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

inline WsLayout make_layout(const Shape &s) {
    WsLayout L{};
    size_t o = align256(sizeof(WsHeader));
    const size_t P = size_t(s.P);
    L.route_cnt = o; o = align256(o + 4 * P);
    L.sel_ready = o; o = align256(o + 4 * P);
    L.part_cnt = o;  o = align256(o + 4 * P);
    L.zrec = o;      o = align256(o + 16 * P * size_t(s.k > 0 ? s.k : 1));
    const size_t nc = P * size_t(s.n_rc) * size_t(s.kc > 0 ? s.kc : 1);
    L.cand_key = o;  o = align256(o + 8 * nc);
    L.cand_idx = o;  o = align256(o + 4 * nc);
    L.cand_len = o;  o = align256(o + 4 * nc);
    L.cand_off = o;  o = align256(o + 8 * nc);
    L.cand_cnt = o;  o = align256(o + 4 * P * size_t(s.n_rc));
    L.cand_lg = o;   o = align256(o + 4 * nc * size_t(s.G));
    const size_t ns = P * size_t(s.n_slots) * size_t(s.G);
    L.part_ml = o;   o = align256(o + 8 * ns);
    L.part_o = o;    o = align256(o + 4 * ns * size_t(s.d));
    L.total = o;
    return L;
}

// Everything a launch needs; passed by value as the kernel argument.
struct Params {
    int32_t mode;
    int32_t B, Hq, Hkv, r, k, A_max, M_max;
    int32_t n_rc, n_ac, kc, n_slots;
    int32_t slot_route0, slot_losers, slot_zoom0;   // first slot of each partial kind
    int32_t end_route, end_anchor, end_zoom;        // item-index ends of each item kind
    int32_t grid;                                   // workgroups in the launch
    int32_t merger;                                 // 1: one workgroup per pair merges the
                                                    // candidates (route mode, or too many
                                                    // candidates for per-item ranking)
    int32_t out_f32;                                // 1: out is float, 0: bf16
    int32_t zoom_impl;
    double scale;                                   // softmax scale (routing score)
    float scale_log2;                               // scale * log2(e): scores in base-2 units
    // cache
    const void *q, *anchor_k, *anchor_v;
    const int32_t *n_anchors;
    const void *sum_k, *sum_v;
    const int32_t *n_spans, *span_len;
    const double *span_logsize;
    const unsigned char *factors;
    int64_t factors_bytes;
    const int64_t *block_off;
    // caller buffers
    int32_t *sel_out;
    float *logits_out;
    const int32_t *sel_in;
    const float *logits_in;
    void *out;
    // workspace
    WsHeader *hdr;
    uint32_t *route_cnt, *sel_ready, *part_cnt;
    int4 *zrec;
    uint64_t *cand_key;
    int32_t *cand_idx, *cand_len, *cand_cnt;
    int64_t *cand_off;
    float *cand_lg;
    float *part_ml, *part_o;
};

// Launchers (sekv_kernels.hip).  Return the HIP error of the launch.
hipError_t launch_step(const Params &p, int dtype, int head_dim, int group, hipStream_t stream);
hipError_t launch_zero(void *ptr, size_t bytes, hipStream_t stream);
int resident_workgroups(int dtype, int head_dim, int group);

}  // namespace sekv
