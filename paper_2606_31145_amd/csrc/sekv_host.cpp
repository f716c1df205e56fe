// Host-only logic of the library (see sekv_host.h).  No HIP runtime calls.
#include "sekv_host.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

namespace sekv {

namespace {
thread_local char g_err[512] = "";

bool misaligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; }

// finite check of n stored values (bf16 bit patterns or float32)
bool all_finite(const void *p, size_t n, int dtype, size_t *bad) {
    if (dtype == SEKV_BF16) {
        const uint16_t *u = static_cast<const uint16_t *>(p);
        for (size_t i = 0; i < n; ++i)
            if ((u[i] & 0x7F80u) == 0x7F80u) { *bad = i; return false; }
    } else {
        const float *f = static_cast<const float *>(p);
        for (size_t i = 0; i < n; ++i)
            if (!std::isfinite(f[i])) { *bad = i; return false; }
    }
    return true;
}
}  // namespace

const char *last_error() { return g_err; }

sekv_status fail(sekv_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

sekv_status check_dims(const sekv_dims *d) {
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
    if (d->top_k < 0 || d->top_k > kMaxTopK)
        return fail(SEKV_ERR_UNSUPPORTED, "top_k %d not in [0,%d]", d->top_k, kMaxTopK);
    if (d->max_anchors < 0) return fail(SEKV_ERR_INVALID_ARG, "max_anchors < 0");
    if (d->max_spans < 1) return fail(SEKV_ERR_INVALID_ARG, "max_spans < 1");
    if (d->max_span_len < 1) return fail(SEKV_ERR_INVALID_ARG, "max_span_len < 1");
    if (d->max_span_len > kMaxSpanLen)
        return fail(SEKV_ERR_UNSUPPORTED, "max_span_len %d > %d", d->max_span_len, kMaxSpanLen);
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
    if (d->max_spans > kMaxSpans)
        return fail(SEKV_ERR_UNSUPPORTED, "max_spans %d > %d", d->max_spans, kMaxSpans);
    const long long rows = (long long)d->batch * d->n_kv_heads * std::max(d->max_spans, d->max_anchors);
    if (rows > (1ll << 31)) return fail(SEKV_ERR_UNSUPPORTED, "tables too large");
    return SEKV_OK;
}

sekv_status check_cache(const sekv_dims *d, const sekv_cache *c, bool need_factors) {
    if (!c) return fail(SEKV_ERR_INVALID_ARG, "cache is NULL");
    if (d->batch == 0) return SEKV_OK;
    // data rows are read as 16-byte vectors; tables element by element
    struct { const void *p; const char *name; uintptr_t align; } ptrs[] = {
        {c->q, "q", 16}, {c->sum_k, "sum_k", 16}, {c->sum_v, "sum_v", 16},
        {c->n_spans, "n_spans", 4}, {c->span_len, "span_len", 4},
        {c->span_logsize, "span_logsize", 8}, {c->n_anchors, "n_anchors", 4}};
    for (auto &x : ptrs) {
        if (!x.p) return fail(SEKV_ERR_INVALID_ARG, "cache.%s is NULL", x.name);
        if (misaligned(x.p, x.align))
            return fail(SEKV_ERR_INVALID_ARG, "cache.%s not %d-byte aligned", x.name, int(x.align));
    }
    if (d->max_anchors > 0) {
        if (!c->anchor_k || !c->anchor_v)
            return fail(SEKV_ERR_INVALID_ARG, "cache.anchor_k/anchor_v is NULL");
        if (misaligned(c->anchor_k, 16) || misaligned(c->anchor_v, 16))
            return fail(SEKV_ERR_INVALID_ARG, "anchor arrays not 16-byte aligned");
    }
    if (need_factors && d->top_k > 0) {
        if (!c->factors || !c->block_off)
            return fail(SEKV_ERR_INVALID_ARG, "cache.factors/block_off is NULL");
        if (misaligned(c->factors, 16) || misaligned(c->block_off, 8))
            return fail(SEKV_ERR_INVALID_ARG, "factor arena not 16-byte or offsets not 8-byte aligned");
        if (c->factors_bytes <= 0) return fail(SEKV_ERR_INVALID_ARG, "factors_bytes <= 0");
    }
    if (misaligned(c->block_rank, 4)) return fail(SEKV_ERR_INVALID_ARG, "cache.block_rank not 4-byte aligned");
    return SEKV_OK;
}

size_t block_bytes(const sekv_dims &d, int L, int rk, int rv) {
    const size_t e = size_t(elem_bytes(d.dtype));
    auto a16 = [](size_t x) { return (x + 15) & ~size_t(15); };
    auto side = [&](int r) {
        return a16(size_t(L) * r * e) + a16(size_t(r) * e) + a16(size_t(r) * d.head_dim * e);
    };
    return side(rk) + side(rv);
}

size_t block_bytes(const sekv_dims &d, int L) { return block_bytes(d, L, d.rank, d.rank); }

bool block_ranks(const sekv_dims &d, const int32_t *table, size_t i, int *rk, int *rv) {
    if (!table) {
        *rk = *rv = d.rank;
        return true;
    }
    const uint32_t w = uint32_t(table[i]);
    *rk = int(w & 0xFFFFu);
    *rv = int(w >> 16);
    const int gran = 16 / elem_bytes(d.dtype);
    auto ok = [&](int r) { return r >= gran && r <= d.rank && r % gran == 0; };
    return ok(*rk) && ok(*rv);
}

sekv_status validate_cache(const sekv_dims *d, const sekv_cache *c) {
    sekv_status st = check_dims(d);
    if (st != SEKV_OK) return st;
    st = check_cache(d, c, true);
    if (st != SEKV_OK) return st;
    const int B = d->batch, Hq = d->n_q_heads, Hkv = d->n_kv_heads, D = d->head_dim;
    const int A_max = d->max_anchors, M = d->max_spans, r = d->rank;
    const size_t e = size_t(elem_bytes(d->dtype));
    const unsigned char *q = static_cast<const unsigned char *>(c->q);
    size_t bad = 0;
    for (int b = 0; b < B; ++b) {
        const int A = c->n_anchors[b], m = c->n_spans[b];
        if (A < 0 || A > A_max) return fail(SEKV_ERR_INVALID_ARG, "n_anchors[%d] = %d outside [0, %d]", b, A, A_max);
        if (m < 0 || m > M) return fail(SEKV_ERR_INVALID_ARG, "n_spans[%d] = %d outside [0, %d]", b, m, M);
        if (A + m < 1) return fail(SEKV_ERR_INVALID_ARG, "sequence %d has no anchors and no spans", b);
        if (!all_finite(q + size_t(b) * Hq * D * e, size_t(Hq) * D, d->dtype, &bad))
            return fail(SEKV_ERR_INVALID_ARG, "q of sequence %d: value %zu not finite", b, bad);
        for (int S = 0; S < m; ++S) {
            const int L = c->span_len[size_t(b) * M + S];
            if (L < 1 || L > d->max_span_len)
                return fail(SEKV_ERR_INVALID_ARG, "span_len[%d][%d] = %d outside [1, %d]", b, S, L, d->max_span_len);
            const double ls = c->span_logsize[size_t(b) * M + S], want = std::log(double(L));
            if (!(std::fabs(ls - want) <= 1e-12 * std::max(1.0, want)))
                return fail(SEKV_ERR_INVALID_ARG, "span_logsize[%d][%d] = %.17g is not ln(%d)", b, S, ls, L);
        }
        for (int g = 0; g < Hkv; ++g) {
            const size_t pr = size_t(b) * Hkv + g;
            if (A > 0) {
                const unsigned char *ak = static_cast<const unsigned char *>(c->anchor_k) + pr * A_max * D * e;
                const unsigned char *av = static_cast<const unsigned char *>(c->anchor_v) + pr * A_max * D * e;
                if (!all_finite(ak, size_t(A) * D, d->dtype, &bad) || !all_finite(av, size_t(A) * D, d->dtype, &bad))
                    return fail(SEKV_ERR_INVALID_ARG, "anchors of (%d, %d): a value is not finite", b, g);
            }
            if (m > 0) {
                const unsigned char *sk = static_cast<const unsigned char *>(c->sum_k) + pr * M * D * e;
                const unsigned char *sv = static_cast<const unsigned char *>(c->sum_v) + pr * M * D * e;
                if (!all_finite(sk, size_t(m) * D, d->dtype, &bad) || !all_finite(sv, size_t(m) * D, d->dtype, &bad))
                    return fail(SEKV_ERR_INVALID_ARG, "summaries of (%d, %d): a value is not finite", b, g);
            }
            if (d->top_k == 0) continue;
            for (int S = 0; S < m; ++S) {
                const int L = c->span_len[size_t(b) * M + S];
                const int64_t off = c->block_off[pr * M + S];
                int rk = r, rv = r;
                if (!block_ranks(*d, c->block_rank, pr * M + S, &rk, &rv))
                    return fail(SEKV_ERR_INVALID_ARG,
                                "block (%d, %d, %d): ranks (%d, %d) not multiples of %d in [%d, %d]", b, g, S, rk,
                                rv, int(16 / e), int(16 / e), r);
                const int64_t n = int64_t(block_bytes(*d, L, rk, rv));
                if (off < 0 || (off & 15) || off + n > c->factors_bytes)
                    return fail(SEKV_ERR_INVALID_ARG,
                                "block (%d, %d, %d) at %lld (+%lld bytes) outside the %lld-byte arena or misaligned",
                                b, g, S, (long long)off, (long long)n, (long long)c->factors_bytes);
                const unsigned char *blk = static_cast<const unsigned char *>(c->factors) + off;
                const size_t vals = (size_t(L) + 1 + size_t(D)) * size_t(rk + rv);
                if (!all_finite(blk, vals, d->dtype, &bad))
                    return fail(SEKV_ERR_INVALID_ARG, "factor block (%d, %d, %d): value %zu not finite", b, g, S, bad);
            }
        }
    }
    return SEKV_OK;
}

sekv_status plan_tier_sequence(const TierPlanIn &in, TierPlan *out) {
    const sekv_dims &d = *in.dims;
    const int Hkv = d.n_kv_heads, k = d.top_k, M = d.max_spans;
    struct Blk { int64_t src, len; int g, s; };
    std::vector<Blk> blks;
    blks.reserve(size_t(Hkv) * size_t(k > 0 ? k : 1));
    for (int g = 0; g < Hkv; ++g)
        for (int j = 0; j < k; ++j) {
            const int s = in.sel[size_t(g) * k + j];
            if (s < 0 || s >= M) continue;
            const int L = in.span_len[s];
            const int64_t off = in.block_off[size_t(g) * M + s];
            if (L < 1 || L > d.max_span_len)
                return fail(SEKV_ERR_INVALID_ARG, "span (%d, %d) has length %d", in.b, s, L);
            int rk = d.rank, rv = d.rank;
            if (!block_ranks(d, in.block_rank, size_t(g) * M + s, &rk, &rv))
                return fail(SEKV_ERR_INVALID_ARG, "host block (%d, %d, %d) has ranks (%d, %d)", in.b, g, s, rk, rv);
            const int64_t len = int64_t(block_bytes(d, L, rk, rv));
            if (off < 0 || (off & 15) || off > in.arena_bytes - len)
                return fail(SEKV_ERR_INVALID_ARG, "host block (%d, %d, %d) outside the arena", in.b, g, s);
            blks.push_back({off, len, g, s});
        }
    // staging of the sequence: its blocks packed in arena order (each on a 256-byte
    // boundary), so blocks that are neighbours in the arena are neighbours in staging
    std::sort(blks.begin(), blks.end(), [](const Blk &x, const Blk &y) {
        return x.src != y.src ? x.src < y.src : (x.g != y.g ? x.g < y.g : x.s < y.s);
    });
    out->runs.clear();
    out->off_set.clear();
    out->bytes = 0;
    if (out->off.size() != size_t(Hkv) * M) out->off.assign(size_t(Hkv) * M, 0);
    int64_t pos = in.region;
    const int64_t end = in.region + in.region_bytes;
    std::vector<int64_t> slot(blks.size());
    for (size_t i = 0; i < blks.size(); ++i) {
        // a span selected by two heads of the same sequence shares one block only if the
        // arena says so (equal offsets); each selection keeps its own staging copy
        slot[i] = pos;
        pos += int64_t(align256(size_t(blks[i].len)));
        if (pos > end) return fail(SEKV_ERR_INVALID_ARG, "staging region of sequence %d overflows", in.b);
        out->off[size_t(blks[i].g) * M + blks[i].s] = slot[i];
        out->off_set.push_back(int32_t(size_t(blks[i].g) * M + blks[i].s));
    }
    for (size_t i = 0; i < blks.size();) {
        size_t j = i + 1;
        while (j < blks.size() &&
               blks[j].src == blks[j - 1].src + int64_t(align256(size_t(blks[j - 1].len))))
            ++j;
        const int64_t len = (blks[j - 1].src - blks[i].src) + blks[j - 1].len;
        out->runs.push_back({blks[i].src, slot[i], len});
        out->bytes += len;
        i = j;
    }
    return SEKV_OK;
}

uint64_t layout_key(const Shape &s) {
    const int64_t f[] = {s.B, s.Hq, s.Hkv, s.d, s.k, s.A_max, s.M_max, s.n_rc, s.kc, s.n_cand, s.n_zi};
    uint64_t h = 1469598103934665603ull;      // FNV-1a over the shape fields
    for (int64_t v : f) {
        h ^= uint64_t(v);
        h *= 1099511628211ull;
    }
    return h == WsTracker::kKeyZeroed ? 1 : h;
}

WsRecord *WsTracker::find(uintptr_t ws) {
    for (auto &r : rec_)
        if (r.stamp && r.ws == ws) return &r;
    return nullptr;
}

WsRecord *WsTracker::slot(uintptr_t ws) {
    WsRecord *r = find(ws);
    if (r) return r;
    WsRecord *old = &rec_[0];
    for (auto &x : rec_) {
        if (!x.stamp) return &x;
        if (x.stamp < old->stamp) old = &x;
    }
    return old;
}

void WsTracker::zeroed(uintptr_t ws, size_t bytes) {
    WsRecord *r = slot(ws);
    *r = WsRecord{ws, bytes, kKeyZeroed, 0, ++clock_};
}

bool WsTracker::before_launch(uintptr_t ws, size_t bytes, uint64_t key, uint64_t n) {
    WsRecord *r = find(ws);
    const bool zero = !r || r->bytes != bytes || (r->key != key && r->key != kKeyZeroed) ||
                      r->launches + n >= kMaxLaunchesPerZero;
    if (zero) {
        if (!r) r = slot(ws);
        *r = WsRecord{ws, bytes, key, 0, 0};
    }
    r->key = key;
    r->launches += n;
    r->stamp = ++clock_;
    return zero;
}


// ---- prefill-side builder: dims check and the factor arena's layout -----------------

sekv_status check_build_dims(const sekv_build_dims *d) {
    if (!d) return fail(SEKV_ERR_INVALID_ARG, "build dims is NULL");
    if (d->batch < 0 || d->n_kv_heads < 1 || d->max_tokens < 1)
        return fail(SEKV_ERR_INVALID_ARG, "batch/n_kv_heads/max_tokens out of range");
    if (d->head_dim != 64 && d->head_dim != 128) return fail(SEKV_ERR_UNSUPPORTED, "head_dim %d", d->head_dim);
    if (d->dtype != SEKV_BF16 && d->dtype != SEKV_F32) return fail(SEKV_ERR_UNSUPPORTED, "dtype %d", d->dtype);
    const int gran = 16 / elem_bytes(d->dtype);
    if (d->rank < gran || d->rank > 40 || d->rank % gran)
        return fail(SEKV_ERR_UNSUPPORTED, "rank %d: a multiple of %d in [%d, 40]", d->rank, gran, gran);
    if (d->sketch < d->rank || d->sketch > 40 || (d->sketch & 1))
        return fail(SEKV_ERR_UNSUPPORTED, "sketch %d: even, in [rank, 40]", d->sketch);
    if (d->min_span < 2) return fail(SEKV_ERR_INVALID_ARG, "min_span %d < 2", d->min_span);
    if (d->window < 0) return fail(SEKV_ERR_INVALID_ARG, "window < 0");
    if (d->sweeps < 1 || d->sweeps > 32) return fail(SEKV_ERR_INVALID_ARG, "sweeps %d outside [1, 32]", d->sweeps);
    if (d->power < 0 || d->power > 4) return fail(SEKV_ERR_INVALID_ARG, "power %d outside [0, 4]", d->power);
    if (d->reserved != 0) return fail(SEKV_ERR_INVALID_ARG, "reserved field is not 0");
    if (!(d->alpha == d->alpha)) return fail(SEKV_ERR_INVALID_ARG, "alpha is NaN");
    return SEKV_OK;
}

int64_t build_layout(const sekv_build_dims *dims, int32_t max_spans, const int32_t *n_spans,
                     const int32_t *span_len, int64_t *block_off, int32_t *block_rank) {
    if (check_build_dims(dims) != SEKV_OK) return -1;
    if (max_spans < 1 || !n_spans || !span_len || !block_off || !block_rank) {
        fail(SEKV_ERR_INVALID_ARG, "NULL argument or max_spans < 1");
        return -1;
    }
    const int B = dims->batch, Hkv = dims->n_kv_heads, N = dims->max_tokens, d = dims->head_dim;
    const int e = elem_bytes(dims->dtype), gran = 16 / e;
    int64_t pos = 0;
    for (int b = 0; b < B; ++b) {
        const int m = n_spans[b];
        if (m < 0 || m > max_spans || m > N) {
            fail(SEKV_ERR_INVALID_ARG, "n_spans[%d] = %d outside [0, %d]", b, m, max_spans);
            return -1;
        }
        for (int g = 0; g < Hkv; ++g)
            for (int S = 0; S < max_spans; ++S) {
                const size_t i = (size_t(b) * Hkv + g) * max_spans + S;
                block_off[i] = 0;
                block_rank[i] = 0;
                if (S >= m) continue;
                const int L = span_len[size_t(b) * N + S];
                if (L < 1 || L > N) {
                    fail(SEKV_ERR_INVALID_ARG, "span_len[%d][%d] = %d", b, S, L);
                    return -1;
                }
                int r = L < d ? L : d;
                if (r > dims->rank) r = dims->rank;
                const int rs = (r + gran - 1) / gran * gran;
                block_off[i] = pos;
                block_rank[i] = rs | (rs << 16);
                pos += int64_t((2 * int64_t(L + 1 + d) * rs * e + 255) / 256 * 256);
            }
    }
    return pos > 0 ? pos : 256;
}

}  // namespace sekv
