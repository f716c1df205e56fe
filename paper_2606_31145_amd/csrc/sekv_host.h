// Host-only logic of the library: argument validation, the host-side cache check, the
// copy plan of the pinned-host tier and the workspace-state bookkeeping.  Nothing here
// calls the HIP runtime, so this part also builds and runs under the address and
// undefined-behaviour sanitizers on a machine without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "sekv.h"
#include "sekv_internal.h"

namespace sekv {

// Thread-local error message (sekv_last_error) and the helpers that set it.
const char *last_error();
sekv_status fail(sekv_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

sekv_status check_dims(const sekv_dims *d);
// Pointer checks of a cache (null, alignment); need_factors: the call zooms.
sekv_status check_cache(const sekv_dims *d, const sekv_cache *c, bool need_factors);

// Bytes of one span block of length L: U|sigma|Vt for keys, then values, every segment
// 16-byte aligned (the ranks and head_dim in use keep them so); without ranks, both
// sides have dims.rank.
size_t block_bytes(const sekv_dims &d, int L);
size_t block_bytes(const sekv_dims &d, int L, int rk, int rv);
// Ranks of a block from its rank-table word (r_K | r_V << 16), or dims.rank for both
// when there is no table.  False when a rank is not a multiple of 16 / element bytes in
// [that, dims.rank].
bool block_ranks(const sekv_dims &d, const int32_t *table, size_t i, int *rk, int *rv);

// Check a cache from HOST copies of its arrays (every pointer in `c` is a host pointer,
// factors_bytes the arena size): the device-side preconditions of the step calls.
sekv_status validate_cache(const sekv_dims *d, const sekv_cache *c);

// ---- pinned-host tier: the copies of one sequence's selected blocks -----------------
struct TierRun {
    int64_t src;      // byte offset in the host arena
    int64_t dst;      // byte offset in device staging
    int64_t bytes;
};
struct TierPlanIn {
    const sekv_dims *dims;
    int b;                        // sequence
    const int32_t *sel;           // [Hkv][k] selection of sequence b (host)
    const int32_t *span_len;      // [M] |S| of sequence b (host)
    const int64_t *block_off;     // [Hkv][M] arena offsets of sequence b's blocks (host)
    int64_t arena_bytes;
    int64_t region;               // first staging byte of sequence b
    int64_t region_bytes;         // staging bytes reserved for sequence b
    const int32_t *block_rank = nullptr;  // [Hkv][M] ranks of sequence b's blocks (host), or null
};
struct TierPlan {
    std::vector<TierRun> runs;    // contiguous runs, in arena order
    std::vector<int64_t> off;     // [Hkv][M]: staging offset of each selected block (else untouched)
    std::vector<int32_t> off_set; // indices into off that were set
    int64_t bytes = 0;
};
// Pack the selected blocks of sequence b into its staging region in arena order (256-byte
// aligned), merging blocks that are neighbours in the arena into one run.  Fails with
// SEKV_ERR_INVALID_ARG for a block outside the arena or a plan that would overflow the
// region.
sekv_status plan_tier_sequence(const TierPlanIn &in, TierPlan *out);
// ---- workspace state (see sekv_api.cpp) -----------------------------------------------
uint64_t layout_key(const Shape &s);

struct WsRecord { uintptr_t ws; size_t bytes; uint64_t key; uint64_t launches; uint64_t stamp; };
class WsTracker {
   public:
    static constexpr int kRecords = 256;
    static constexpr uint64_t kKeyZeroed = 0;
    static constexpr uint64_t kMaxLaunchesPerZero = 1ull << 31;
    // The workspace was just zeroed.
    void zeroed(uintptr_t ws, size_t bytes);
    // n launches of layout `key` are about to be enqueued on ws; returns true when the
    // workspace must be zeroed first (the record then counts from the zeroing).
    bool before_launch(uintptr_t ws, size_t bytes, uint64_t key, uint64_t n);

   private:
    WsRecord *find(uintptr_t ws);
    WsRecord *slot(uintptr_t ws);
    WsRecord rec_[kRecords] = {};
    uint64_t clock_ = 0;
};

// ---- prefill-side builder ------------------------------------------------------------
sekv_status check_build_dims(const sekv_build_dims *d);
// The factor arena of a segmentation from host copies of n_spans [B] and span_len
// [B][max_tokens] (sekv_build_layout): block_off and block_rank [B][Hkv][max_spans];
// returns the arena bytes, or -1 with the error message set.
int64_t build_layout(const sekv_build_dims *dims, int32_t max_spans, const int32_t *n_spans,
                     const int32_t *span_len, int64_t *block_off, int32_t *block_rank);

}  // namespace sekv
