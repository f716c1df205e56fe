// Launch structures of the prefill-side builder (sekv_build.hip, sekv_build_api.cpp),
// kept apart from the decode step's internals.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace sekv {

// Prefill-side builder (sekv_build.hip).
struct SegArgs {
    const float *surprisal;            // [B][N]
    const int32_t *n_tokens;           // [B]
    int32_t *n_anchors, *anchor_idx;   // [B], [B][N]
    int32_t *n_spans, *span_start, *span_len;   // [B], [B][N], [B][N]
    unsigned char *ws_flag, *ws_inspan;         // [B][N] scratch
    int32_t *ws_pos;                   // [B][N + 2] scratch
    double alpha;
    int32_t N, min_span, window;
};
struct BuildArgs {
    const void *keys, *values;         // [B][Hkv][N][d]
    const float *surprisal;            // [B][N]
    const int32_t *n_tokens;           // [B]
    const int32_t *n_anchors, *anchor_idx, *n_spans, *span_start, *span_len_seg;
    const float *omega;                // [d][l]
    void *anchor_k, *anchor_v;         // [B][Hkv][A_max][d]
    void *sum_k, *sum_v;               // [B][Hkv][M_max][d]
    int32_t *span_len_out;             // [B][M_max]
    double *span_logsize;              // [B][M_max]
    void *factors;
    int64_t factors_bytes;
    const int64_t *block_off;          // [B][Hkv][M_max]
    int32_t *error;                    // device error word (out-of-arena blocks, bad tables)
    int32_t Hkv, N, d, elem, R, l, sweeps, power, A_max, M_max;
    int64_t *trace;                    // diagnostic builds: [trace_items][kTraceSlots] or null
    int64_t trace_items;
};

// The phase-trace buffer attached by sekv_phase_trace (null unless a trace build has one).
int64_t *trace_buffer(size_t *bytes);

hipError_t launch_segment(const SegArgs &a, int batch, hipStream_t stream);
hipError_t launch_build(const BuildArgs &a, int batch, hipStream_t stream);

}  // namespace sekv
