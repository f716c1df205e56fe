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
constexpr int kRouteChunk = 128;   // spans per routing work item
constexpr int kZoomBlock = 512;    // tokens of a zoomed span scored per LDS pass
constexpr int kMaxTopK = 64;
constexpr int kMergeBuf = 512;     // candidates ranked in LDS by one workgroup
constexpr int kMaxSpans = 65536;   // max_spans limit (span indices and record sizes)
constexpr int kMaxSpanLen = 1 << 20; // max_span_len limit
constexpr int kShareTarget = 512;  // share items per launch above which a share item
                                   // zooms several selection slots
constexpr int kRoundItems = 512;   // items a launch starts at once on a 256-CU device at
                                   // two workgroups per CU (used only to split the work;
                                   // a constant, so the split never depends on the device)

enum Mode : int32_t { kModeRoute = 0, kModeAttend = 1, kModeFused = 2 };

// Learned-routing selection (sekv_gate.hip): one workgroup scores a chunk of spans,
// a power of two >= kGateMinChunk chosen so that a pair's candidates fit one LDS sort.
constexpr int kGateMinChunk = 256;
constexpr int kGateMaxCand = 2048;  // candidates (chunks x k) of a pair, and the largest chunk
constexpr int kGateMaxDr = 64;      // largest routing dimension d'
constexpr int kGateMaxG = 8;        // largest Hq / Hkv

// Phase trace (diagnostic builds compiled with SEKV_PHASE_TRACE): per work item,
// kTraceSlots int64 words; slot 0 holds the item's descriptor, the others the
// s_memrealtime value (100 MHz) at the phase marks listed with the kernel.
constexpr int kTraceSlots = 16;

// Device error bits (workspace header word `error`).
enum : int32_t { kErrSpinTimeout = 1, kErrBlockRange = 2, kErrSelRange = 4 };

// Fields of a tagged candidate record (one 64-bit word each, 32-bit payload).
enum : int32_t { kCandKeyHi = 0, kCandKeyLo, kCandIdx, kCandLen, kCandOffLo, kCandOffHi, kCandFields };

// Workspace header.  `epoch` is the tag of the next launch: that launch marks the words
// it publishes with it, and its last workgroup out advances it (skipping 0, the value
// of never-written words; initialisation sets 1) and zeroes every counter it used.
struct WsHeader {
    uint32_t unused0;
    uint32_t exit_count;
    int32_t error;
    uint32_t epoch;
    uint32_t pad[60];
};

// Byte offsets of the workspace sections for one dims.
struct WsLayout {
    size_t route_cnt, sel_ready, part_cnt;    // uint32 [P]
    size_t claim;                             // uint32 [P][n_rc]: tag of the launch that claimed a chunk
    size_t zrec;                              // int32x4 [P][k]: span, |S|, offset lo/hi
    size_t cand;                              // tagged uint64 [kCandFields][P][n_cand]
    size_t tlg;                               // tagged uint64 [P][G][M_max]: base-2 logits
    size_t part_ml;                           // float pairs (m, l) [P][n_zi][G]
    size_t part_o;                            // float pairs [P][n_zi][G][d/2]
    size_t gate_cnt;                          // uint32 [P]: learned-routing chunks done
    size_t gate_cand;                         // uint64 pairs [P][g_nrc][k]: chunk candidates
    size_t total;
};

struct Shape {
    int B, Hq, Hkv, G, d, r, k, A_max, M_max, L_max;
    int P;        // B * Hkv pairs
    int n_rc;     // routing chunks per pair
    int kc;       // candidates kept per routing chunk = min(k, kRouteChunk)
    int n_cand;   // candidates per pair = n_rc * kc
    int n_zi;     // share items (and partials) per pair; share item j zooms the spans
                  // of ranks j, j + n_zi, ... below k
    int g_cr;     // learned routing: spans per chunk (power of two)
    int g_nrc;    // learned routing: chunks per pair
};

inline int elem_bytes(int dtype) { return dtype == SEKV_BF16 ? 2 : 4; }

inline Shape make_shape(const sekv_dims &d) {
    Shape s{};
    s.B = d.batch; s.Hq = d.n_q_heads; s.Hkv = d.n_kv_heads; s.G = s.Hq / s.Hkv;
    s.d = d.head_dim; s.r = d.rank; s.k = d.top_k;
    s.A_max = d.max_anchors; s.M_max = d.max_spans; s.L_max = d.max_span_len;
    s.P = s.B * s.Hkv;
    s.n_rc = (s.M_max + kRouteChunk - 1) / kRouteChunk;
    s.kc = s.k < kRouteChunk ? s.k : kRouteChunk;
    s.n_cand = s.n_rc * s.kc;
    // one share item per selection slot while the pairs leave room for that; with many
    // pairs, fewer items per pair so the launch runs about one round of share items.
    // The split depends only on the shapes, so results are the same bits on any device.
    const int P1 = s.P > 0 ? s.P : 1;
    const int fit = (kShareTarget + P1 - 1) / P1;
    s.n_zi = s.k > 1 ? s.k : 1;
    if (s.n_zi > fit) s.n_zi = fit;
    const int kk = s.k > 1 ? s.k : 1;
    s.g_cr = kGateMinChunk;
    while (s.g_cr < kGateMaxCand && ((s.M_max + s.g_cr - 1) / s.g_cr) * kk > kGateMaxCand) s.g_cr *= 2;
    s.g_nrc = (s.M_max + s.g_cr - 1) / s.g_cr;
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
    L.claim = o;     o = align256(o + 4 * P * size_t(s.n_rc));
    L.zrec = o;      o = align256(o + 16 * P * size_t(s.k > 0 ? s.k : 1));
    L.cand = o;      o = align256(o + 8 * size_t(kCandFields) * P * size_t(s.n_cand > 0 ? s.n_cand : 1));
    L.tlg = o;       o = align256(o + 8 * P * size_t(s.G) * size_t(s.M_max));
    const size_t ns = P * size_t(s.n_zi) * size_t(s.G);
    L.part_ml = o;   o = align256(o + 8 * ns);
    L.part_o = o;    o = align256(o + 4 * ns * size_t(s.d));
    L.gate_cnt = o;  o = align256(o + 4 * P);
    L.gate_cand = o; o = align256(o + 16 * P * size_t(s.g_nrc) * size_t(s.k > 0 ? s.k : 1));
    L.total = o;
    return L;
}

// Everything a launch needs; passed by value as the kernel argument.
struct Params {
    int32_t mode;
    int32_t B, Hq, Hkv, r, k, A_max, M_max;
    int32_t n_rc, kc, n_cand, n_zi;
    int32_t end_route, end_share;                   // item-index ends of each item kind
    int32_t n_early;                                // share slots j < n_early take the anchors
    int32_t grid;                                   // workgroups in the launch
    int32_t merger;                                 // 1: one workgroup per pair merges the
                                                    // candidates (route mode, or more than
                                                    // kMergeBuf candidates)
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
    const int32_t *block_rank;                      // r_K | r_V << 16 per block, or null
    // caller buffers
    int32_t *sel_out;
    float *logits_out;
    const int32_t *sel_in;
    const float *logits_in;
    void *out;
    // workspace
    WsHeader *hdr;
    uint32_t *route_cnt, *sel_ready, *part_cnt;
    uint32_t *claim;
    int4 *zrec;
    uint64_t *cand;
    uint64_t *tlg;
    uint64_t *part_ml, *part_o;
    int64_t *trace;                                 // [end_share][kTraceSlots] or null
};

// Launch parameters of the learned-routing selection kernel (sekv_gate.hip).
struct GateParams {
    int32_t B, Hq, Hkv, G, d, dr, k, M_max;
    int32_t cr, n_rc;                  // spans per chunk (power of two), chunks per pair
    int64_t budget;                    // expanded tokens allowed per pair
    double scale_r;                    // 1 / sqrt(d')
    const void *q, *proj, *sum_route;
    const int32_t *n_spans, *span_len;
    const double *span_logsize, *thr;
    int32_t *sel;                      // [B][Hkv][k]
    double *gate_out;                  // [B][Hq][M_max] or null
    uint32_t *cnt;                     // [P]
    uint64_t *cand;                    // [P][n_rc][k] x 2 words
};

// Bytes a tier gather workgroup moves at a time.
constexpr int kGatherChunk = 32768;

// Device-planned tier gather of one sequence (sekv_tier.hip): selection slot (g, j) of
// the sequence is copied to staging bytes [slot0 + (g k + j) slot_bytes, ...).
struct TierGatherArgs {
    const unsigned char *arena;        // device mapping of the pinned host arena
    unsigned char *staging;
    const int32_t *sel;                // [Hkv][k] (device)
    const int32_t *span_len;           // [M] (device)
    const int64_t *block_off;          // [Hkv][M] arena offsets (device)
    int64_t *stage_off;                // [Hkv][M] staging offsets, written for selected spans
    unsigned long long *stats;         // [2]: bytes and blocks moved (accumulated)
    int32_t *error;                    // workspace error word (out-of-arena blocks)
    const int32_t *block_rank;         // [Hkv][M] r_K | r_V << 16 (device), or null: r for both
    int64_t arena_bytes, slot0, slot_bytes;
    int32_t Hkv, k, M, r, d, elem, max_span_len, chunks_per_slot;
};

// One pass of the layered tier over every sequence (sekv_tier.hip).  prefetch = 1: copy
// the blocks of `sel` (the previous layer's selection) into the prefetch slots and record
// which span each slot holds in pf_span.  prefetch = 0: for every selected span, point
// stage_off at its prefetch slot when pf_span holds it (use_pf), else copy it into its
// miss slot.
struct LayerCopyArgs {
    const unsigned char *arena;        // device mapping of the layer's pinned arena
    unsigned char *staging;            // the layer buffer: prefetch region, then miss region
    const int32_t *sel;                // [B][Hkv][k]
    const int32_t *span_len;           // [B][M]
    const int64_t *block_off;          // [B][Hkv][M] arena offsets (device)
    const int32_t *block_rank;         // [B][Hkv][M] or null
    int64_t *stage_off;                // [B][Hkv][M]
    int32_t *pf_span;                  // [B][Hkv][k]
    unsigned long long *stats;         // [4]: miss bytes, miss blocks, prefetch bytes, blocks
    int32_t *error;
    int64_t arena_bytes, slot_bytes, miss0;   // miss0: byte offset of the miss region
    int32_t B, Hkv, k, M, r, d, elem, max_span_len, chunks_per_slot, prefetch, use_pf;
};

// Launchers (sekv_kernels.hip).  Return the HIP error of the launch.
hipError_t launch_step(const Params &p, int dtype, int head_dim, int group, hipStream_t stream);
hipError_t launch_zero(void *ptr, size_t bytes, hipStream_t stream);
hipError_t launch_tier_gather(const TierGatherArgs &a, hipStream_t stream);
hipError_t launch_stats_reset(unsigned long long *stats, hipStream_t stream);
hipError_t launch_layer_copy(const LayerCopyArgs &a, hipStream_t stream);
hipError_t launch_stats_reset4(unsigned long long *stats, hipStream_t stream);
hipError_t launch_gate(const GateParams &g, int dtype, hipStream_t stream);
int resident_workgroups(int dtype, int head_dim, int group);

// The fused step on a given workspace, with every host check (sekv_api.cpp).
sekv_status run_fused_step(const sekv_dims *d, const sekv_cache *c, int32_t *sel, void *out, void *ws,
                           size_t ws_bytes, hipStream_t stream);

}  // namespace sekv
