// Host-only checks of the library's host layer (argument validation, the host-side cache
// check, the pinned-host tier's copy plan, the workspace bookkeeping and the builder's
// dims check and factor-arena layout), built with g++
// under the address and undefined-behaviour sanitizers by tests/test_host_sanitized.py.
// No GPU and no HIP runtime are involved.  Prints "all host checks passed" on success.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "sekv_host.h"

namespace {

int g_fail = 0;
#define CHECK(cond)                                                                   \
    do {                                                                              \
        if (!(cond)) {                                                                \
            std::printf("FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond,         \
                        sekv::last_error());                                          \
            ++g_fail;                                                                 \
        }                                                                             \
    } while (0)

sekv_dims base_dims() {
    sekv_dims d{};
    d.batch = 2; d.n_q_heads = 8; d.n_kv_heads = 2; d.head_dim = 64; d.rank = 8; d.top_k = 3;
    d.max_anchors = 5; d.max_spans = 6; d.max_span_len = 40; d.dtype = SEKV_F32; d.out_dtype = SEKV_F32;
    d.flags = 0; d.softmax_scale = 0.125;
    return d;
}

void test_check_dims() {
    sekv_dims d = base_dims();
    CHECK(sekv::check_dims(&d) == SEKV_OK);
    CHECK(sekv::check_dims(nullptr) == SEKV_ERR_INVALID_ARG);
    struct Case { void (*mut)(sekv_dims &); sekv_status want; } cases[] = {
        {[](sekv_dims &x) { x.batch = -1; }, SEKV_ERR_INVALID_ARG},
        {[](sekv_dims &x) { x.n_q_heads = 6; x.n_kv_heads = 4; }, SEKV_ERR_INVALID_ARG},
        {[](sekv_dims &x) { x.n_q_heads = 12; x.n_kv_heads = 4; }, SEKV_ERR_UNSUPPORTED},
        {[](sekv_dims &x) { x.head_dim = 96; }, SEKV_ERR_UNSUPPORTED},
        {[](sekv_dims &x) { x.rank = 12; }, SEKV_ERR_UNSUPPORTED},
        {[](sekv_dims &x) { x.top_k = 65; }, SEKV_ERR_UNSUPPORTED},
        {[](sekv_dims &x) { x.max_spans = 0; }, SEKV_ERR_INVALID_ARG},
        {[](sekv_dims &x) { x.max_span_len = 0; }, SEKV_ERR_INVALID_ARG},
        {[](sekv_dims &x) { x.max_span_len = (1 << 20) + 1; }, SEKV_ERR_UNSUPPORTED},
        {[](sekv_dims &x) { x.softmax_scale = 0.0; }, SEKV_ERR_INVALID_ARG},
        {[](sekv_dims &x) { x.softmax_scale = INFINITY; }, SEKV_ERR_INVALID_ARG},
        {[](sekv_dims &x) { x.out_dtype = SEKV_BF16; }, SEKV_ERR_UNSUPPORTED},
        {[](sekv_dims &x) { x.flags = 4; }, SEKV_ERR_UNSUPPORTED},
        {[](sekv_dims &x) { x.max_spans = 70000; }, SEKV_ERR_UNSUPPORTED},
    };
    for (auto &c : cases) {
        sekv_dims x = base_dims();
        c.mut(x);
        CHECK(sekv::check_dims(&x) == c.want);
    }
}

// A small host cache laid out as the device cache would be (float32 storage).
struct HostCache {
    sekv_dims d;
    std::vector<float> q, ak, av, sk, sv;
    std::vector<int32_t> n_anchors, n_spans, span_len;
    std::vector<double> logsize;
    std::vector<int64_t> block_off;
    std::vector<unsigned char> arena;
    sekv_cache view() {
        sekv_cache c{};
        c.q = q.data(); c.anchor_k = ak.data(); c.anchor_v = av.data(); c.n_anchors = n_anchors.data();
        c.sum_k = sk.data(); c.sum_v = sv.data(); c.n_spans = n_spans.data(); c.span_len = span_len.data();
        c.span_logsize = logsize.data(); c.factors = arena.data();
        c.factors_bytes = int64_t(arena.size()); c.block_off = block_off.data();
        return c;
    }
};

HostCache make_cache(std::mt19937 &rng) {
    HostCache h;
    h.d = base_dims();
    const sekv_dims &d = h.d;
    const int B = d.batch, Hkv = d.n_kv_heads, D = d.head_dim, A = d.max_anchors, M = d.max_spans;
    std::normal_distribution<float> nd;
    auto fill = [&](std::vector<float> &v, size_t n) { v.resize(n); for (auto &x : v) x = nd(rng); };
    fill(h.q, size_t(B) * d.n_q_heads * D);
    fill(h.ak, size_t(B) * Hkv * A * D);
    fill(h.av, size_t(B) * Hkv * A * D);
    fill(h.sk, size_t(B) * Hkv * M * D);
    fill(h.sv, size_t(B) * Hkv * M * D);
    h.n_anchors = {A, 2};
    h.n_spans = {M, 4};
    h.span_len.assign(size_t(B) * M, 0);
    h.logsize.assign(size_t(B) * M, 0.0);
    std::uniform_int_distribution<int> ld(1, d.max_span_len);
    for (int b = 0; b < B; ++b)
        for (int S = 0; S < h.n_spans[b]; ++S) {
            const int L = ld(rng);
            h.span_len[size_t(b) * M + S] = L;
            h.logsize[size_t(b) * M + S] = std::log(double(L));
        }
    h.block_off.assign(size_t(B) * Hkv * M, 0);
    int64_t total = 0;
    for (int b = 0; b < B; ++b)
        for (int g = 0; g < Hkv; ++g)
            for (int S = 0; S < h.n_spans[b]; ++S) {
                h.block_off[(size_t(b) * Hkv + g) * M + S] = total;
                total += int64_t(sekv::align256(sekv::block_bytes(d, h.span_len[size_t(b) * M + S])));
            }
    h.arena.assign(size_t(total), 0);
    float *f = reinterpret_cast<float *>(h.arena.data());
    for (size_t i = 0; i < h.arena.size() / 4; ++i) f[i] = nd(rng);
    return h;
}

void test_validate_cache(std::mt19937 &rng) {
    {
        HostCache h = make_cache(rng);
        sekv_cache c = h.view();
        CHECK(sekv::validate_cache(&h.d, &c) == SEKV_OK);
    }
    const int M = base_dims().max_spans;
    struct Bad { const char *what; void (*mut)(HostCache &); } bad[] = {
        {"too many anchors", [](HostCache &h) { h.n_anchors[1] = h.d.max_anchors + 1; }},
        {"negative span count", [](HostCache &h) { h.n_spans[0] = -1; }},
        {"too many spans", [](HostCache &h) { h.n_spans[1] = h.d.max_spans + 1; }},
        {"empty sequence", [](HostCache &h) { h.n_anchors[1] = 0; h.n_spans[1] = 0; }},
        {"zero-length span", [](HostCache &h) { h.span_len[2] = 0; }},
        {"over-long span", [](HostCache &h) { h.span_len[1] = h.d.max_span_len + 1; }},
        {"wrong log size", [](HostCache &h) { h.logsize[3] += 1e-6; }},
        {"misaligned block", [](HostCache &h) { h.block_off[1] += 8; }},
        {"block past the arena", [](HostCache &h) { h.block_off[2] = int64_t(h.arena.size()) - 16; }},
        {"negative offset", [](HostCache &h) { h.block_off[0] = -256; }},
        {"NaN query", [](HostCache &h) { h.q[7] = NAN; }},
        {"Inf anchor value", [](HostCache &h) { h.av[3] = INFINITY; }},
        {"NaN summary", [](HostCache &h) { h.sk[5] = NAN; }},
        {"Inf factor", [](HostCache &h) {
             reinterpret_cast<float *>(h.arena.data() + h.block_off[1])[3] = -INFINITY; }},
    };
    (void)M;
    for (auto &x : bad) {
        HostCache h = make_cache(rng);
        x.mut(h);
        sekv_cache c = h.view();
        const sekv_status st = sekv::validate_cache(&h.d, &c);
        if (st != SEKV_ERR_INVALID_ARG) std::printf("  not caught: %s\n", x.what);
        CHECK(st == SEKV_ERR_INVALID_ARG);
    }
    // rows past the counts are never looked at
    {
        HostCache h = make_cache(rng);
        h.ak[((size_t(0) * h.d.n_kv_heads + 1) * h.d.max_anchors + 4) * h.d.head_dim] = NAN;  // b 0, g 1, row 4 < 5
        sekv_cache c = h.view();
        CHECK(sekv::validate_cache(&h.d, &c) == SEKV_ERR_INVALID_ARG);
        HostCache h2 = make_cache(rng);
        const size_t row = (size_t(1) * h2.d.n_kv_heads + 0) * h2.d.max_anchors + 3;      // b 1: 2 anchors
        h2.ak[row * h2.d.head_dim] = NAN;
        c = h2.view();
        CHECK(sekv::validate_cache(&h2.d, &c) == SEKV_OK);
    }
}

void test_tier_plan(std::mt19937 &rng) {
    for (int trial = 0; trial < 300; ++trial) {
        sekv_dims d = base_dims();
        d.batch = 1;
        d.n_kv_heads = 1 + int(rng() % 4);
        d.n_q_heads = d.n_kv_heads * 2;
        d.top_k = 1 + int(rng() % 8);
        d.max_spans = 4 + int(rng() % 40);
        d.max_span_len = 1 + int(rng() % 300);
        d.rank = 8 << int(rng() % 3);
        d.dtype = (rng() & 1) ? SEKV_BF16 : SEKV_F32;
        d.out_dtype = SEKV_F32;
        const int Hkv = d.n_kv_heads, k = d.top_k, M = d.max_spans;
        std::vector<int32_t> len(M);
        for (auto &L : len) L = 1 + int(rng() % d.max_span_len);
        // half of the cases carry per-block ranks (multiples of 16 bytes of elements)
        const bool ranked = (rng() & 1) != 0;
        const int gran = 16 / sekv::elem_bytes(d.dtype);
        std::vector<int32_t> rnk(size_t(Hkv) * M, 0);
        for (auto &w : rnk) {
            const int nmax = d.rank / gran;
            const int rk = gran * (1 + int(rng() % nmax)), rv = gran * (1 + int(rng() % nmax));
            w = rk | (rv << 16);
        }
        auto bsz = [&](int g, int s) {
            if (!ranked) return int64_t(sekv::block_bytes(d, len[s]));
            const int32_t w = rnk[size_t(g) * M + s];
            return int64_t(sekv::block_bytes(d, len[s], w & 0xFFFF, w >> 16));
        };
        std::vector<int64_t> off(size_t(Hkv) * M);
        int64_t pos = 0;
        for (int g = 0; g < Hkv; ++g)
            for (int s = 0; s < M; ++s) {
                off[size_t(g) * M + s] = pos;
                pos += int64_t(sekv::align256(size_t(bsz(g, s))));
            }
        std::vector<int32_t> sel(size_t(Hkv) * k, -1);
        for (int g = 0; g < Hkv; ++g) {
            std::vector<int> perm(M);
            for (int i = 0; i < M; ++i) perm[i] = i;
            std::shuffle(perm.begin(), perm.end(), rng);
            const int take = int(rng() % (k + 1));
            for (int j = 0; j < take && j < M; ++j) sel[size_t(g) * k + j] = perm[j];
        }
        const int64_t slot = int64_t(sekv::align256(sekv::block_bytes(d, d.max_span_len)));
        const int64_t region0 = 4096, region = int64_t(Hkv) * k * slot;
        sekv::TierPlanIn in{&d, 0, sel.data(), len.data(), off.data(), pos, region0, region,
                            ranked ? rnk.data() : nullptr};
        sekv::TierPlan plan;
        CHECK(sekv::plan_tier_sequence(in, &plan) == SEKV_OK);
        // every selected block: its staging slot lies in the region, 256-aligned, and one run
        // maps its arena bytes onto exactly those staging bytes
        int64_t want_bytes = 0;
        std::vector<std::pair<int64_t, int64_t>> slots;
        for (int g = 0; g < Hkv; ++g)
            for (int j = 0; j < k; ++j) {
                const int s = sel[size_t(g) * k + j];
                if (s < 0) continue;
                const int64_t st = plan.off[size_t(g) * M + s];
                const int64_t n = bsz(g, s);
                want_bytes += n;
                CHECK(st >= region0 && st + n <= region0 + region && st % 256 == 0);
                slots.push_back({st, st + n});
                bool covered = false;
                for (const auto &r : plan.runs) {
                    const int64_t src = off[size_t(g) * M + s];
                    if (src >= r.src && src + n <= r.src + r.bytes && r.dst + (src - r.src) == st)
                        covered = true;
                }
                CHECK(covered);
            }
        std::sort(slots.begin(), slots.end());
        for (size_t i = 1; i < slots.size(); ++i) CHECK(slots[i].first >= slots[i - 1].second);
        int64_t run_bytes = 0;
        for (size_t i = 0; i < plan.runs.size(); ++i) {
            run_bytes += plan.runs[i].bytes;
            if (i) CHECK(plan.runs[i].src > plan.runs[i - 1].src);
        }
        CHECK(run_bytes == plan.bytes);
        CHECK(plan.bytes >= want_bytes);            // runs also carry the padding between blocks
        // a block outside the arena, and a region too small, are refused
        if (!plan.runs.empty()) {
            sekv::TierPlanIn bad = in;
            bad.arena_bytes = plan.runs.back().src + plan.runs.back().bytes - 16;
            CHECK(sekv::plan_tier_sequence(bad, &plan) == SEKV_ERR_INVALID_ARG);
            sekv::TierPlanIn small = in;
            small.region_bytes = 255;
            CHECK(sekv::plan_tier_sequence(small, &plan) == SEKV_ERR_INVALID_ARG);
            if (ranked) {
                // a rank off the granule is refused
                int first = -1;
                for (int i = 0; i < Hkv * k && first < 0; ++i)
                    if (sel[size_t(i)] >= 0) first = i;
                std::vector<int32_t> badr = rnk;
                badr[size_t(first / k) * M + sel[size_t(first)]] = (gran + 1) | (gran << 16);
                sekv::TierPlanIn br = in;
                br.block_rank = badr.data();
                CHECK(sekv::plan_tier_sequence(br, &plan) == SEKV_ERR_INVALID_ARG);
            }
        }
    }
}

void test_ws_tracker() {
    sekv::WsTracker t;
    sekv_dims d = base_dims();
    const uint64_t k1 = sekv::layout_key(sekv::make_shape(d));
    d.batch = 3;
    const uint64_t k2 = sekv::layout_key(sekv::make_shape(d));
    CHECK(k1 != k2 && k1 != 0 && k2 != 0);
    CHECK(k1 == sekv::layout_key(sekv::make_shape(base_dims())));
    const uintptr_t ws = 0x100000, ws2 = 0x200000;
    CHECK(t.before_launch(ws, 4096, k1, 1));          // never seen: zero first
    CHECK(!t.before_launch(ws, 4096, k1, 1));         // same layout
    CHECK(t.before_launch(ws, 4096, k2, 1));          // layout changed
    CHECK(!t.before_launch(ws, 4096, k2, 5));
    CHECK(t.before_launch(ws, 8192, k2, 1));          // same address, another size
    t.zeroed(ws2, 4096);
    CHECK(!t.before_launch(ws2, 4096, k1, 1));        // freshly zeroed: any layout
    CHECK(t.before_launch(ws2, 4096, k2, 1));
    CHECK(!t.before_launch(ws2, 4096, k2, sekv::WsTracker::kMaxLaunchesPerZero - 3));
    CHECK(t.before_launch(ws2, 4096, k2, 5));         // the epoch would come round again
    // eviction: after many other workspaces, the record of ws is gone and it is zeroed again
    for (int i = 0; i < 2 * sekv::WsTracker::kRecords; ++i) t.before_launch(0x1000000 + 4096 * uintptr_t(i), 4096, k1, 1);
    CHECK(t.before_launch(ws, 8192, k2, 1));
}


sekv_build_dims base_build_dims() {
    sekv_build_dims d{};
    d.batch = 3; d.n_kv_heads = 2; d.head_dim = 128; d.max_tokens = 700; d.rank = 32; d.sketch = 40;
    d.min_span = 4; d.window = 16; d.sweeps = 8; d.dtype = SEKV_BF16; d.power = 1; d.reserved = 0;
    d.alpha = 1.0;
    return d;
}

// The builder's dims check and the arena layout from random span tables: blocks in (b, g, S)
// order, 256-byte aligned, back to back without overlap, each of the size its span and
// stored rank give, ranks min(|S|, d, R_max) rounded up to the granule, zero entries past
// n_spans[b]; bad tables and arguments rejected.
void test_build_layout(std::mt19937 &rng) {
    sekv_build_dims d = base_build_dims();
    CHECK(sekv::check_build_dims(&d) == SEKV_OK);
    CHECK(sekv::check_build_dims(nullptr) == SEKV_ERR_INVALID_ARG);
    struct Case { int field; int32_t value; sekv_status want; };
    const Case cases[] = {
        {0, -1, SEKV_ERR_INVALID_ARG}, {1, 0, SEKV_ERR_INVALID_ARG}, {2, 96, SEKV_ERR_UNSUPPORTED},
        {3, 0, SEKV_ERR_INVALID_ARG}, {4, 36, SEKV_ERR_UNSUPPORTED}, {4, 48, SEKV_ERR_UNSUPPORTED},
        {5, 30, SEKV_ERR_UNSUPPORTED}, {5, 39, SEKV_ERR_UNSUPPORTED}, {5, 42, SEKV_ERR_UNSUPPORTED},
        {6, 1, SEKV_ERR_INVALID_ARG}, {7, -1, SEKV_ERR_INVALID_ARG}, {8, 0, SEKV_ERR_INVALID_ARG},
        {8, 33, SEKV_ERR_INVALID_ARG}, {9, 7, SEKV_ERR_UNSUPPORTED}, {10, 5, SEKV_ERR_INVALID_ARG},
        {11, 1, SEKV_ERR_INVALID_ARG},
    };
    for (const Case &c : cases) {
        sekv_build_dims x = d;
        int32_t *f[] = {&x.batch, &x.n_kv_heads, &x.head_dim, &x.max_tokens, &x.rank, &x.sketch,
                        &x.min_span, &x.window, &x.sweeps, &x.dtype, &x.power, &x.reserved};
        *f[c.field] = c.value;
        CHECK(sekv::check_build_dims(&x) == c.want);
    }
    {
        sekv_build_dims x = d;
        x.alpha = std::nan("");
        CHECK(sekv::check_build_dims(&x) == SEKV_ERR_INVALID_ARG);
    }
    for (int round = 0; round < 200; ++round) {
        sekv_build_dims x = d;
        x.head_dim = (round & 1) ? 64 : 128;
        x.dtype = (round & 2) ? SEKV_F32 : SEKV_BF16;
        const int e = x.dtype == SEKV_BF16 ? 2 : 4, gran = 16 / e;
        x.rank = gran * (1 + int(rng() % unsigned(40 / gran)));
        x.sketch = std::max(x.rank + (x.rank & 1), 2 * int((x.rank + 1 + rng() % 8) / 2));
        if (x.sketch > 40) x.sketch = 40;
        x.batch = 1 + int(rng() % 3);
        const int B = x.batch, Hkv = x.n_kv_heads, N = x.max_tokens, dd = x.head_dim;
        const int max_spans = 1 + int(rng() % 12);
        std::vector<int32_t> ns(B), len(size_t(B) * N, 0);
        for (int b = 0; b < B; ++b) {
            ns[b] = int(rng() % unsigned(max_spans + 1));
            for (int S = 0; S < ns[b]; ++S) len[size_t(b) * N + S] = 1 + int(rng() % unsigned(N));
        }
        const size_t nb = size_t(B) * Hkv * max_spans;
        std::vector<int64_t> off(nb, -7);
        std::vector<int32_t> rk(nb, -7);
        const int64_t bytes = sekv::build_layout(&x, max_spans, ns.data(), len.data(), off.data(), rk.data());
        CHECK(bytes > 0 && bytes % 256 == 0);
        int64_t pos = 0;
        for (int b = 0; b < B; ++b)
            for (int g = 0; g < Hkv; ++g)
                for (int S = 0; S < max_spans; ++S) {
                    const size_t i = (size_t(b) * Hkv + g) * max_spans + S;
                    if (S >= ns[b]) {
                        CHECK(off[i] == 0 && rk[i] == 0);
                        continue;
                    }
                    const int L = len[size_t(b) * N + S];
                    const int r = std::min(std::min(L, dd), x.rank);
                    const int rs = (r + gran - 1) / gran * gran;
                    CHECK(rk[i] == (rs | (rs << 16)));
                    CHECK(off[i] == pos && off[i] % 256 == 0);
                    const int64_t need = 2 * int64_t(L + 1 + dd) * rs * e;
                    pos += (need + 255) / 256 * 256;
                    CHECK(off[i] + need <= bytes);
                }
        CHECK(bytes == (pos > 0 ? pos : 256));
        // a span longer than the row stride, an empty span, more spans than max_spans
        if (ns[0] > 0) {
            std::vector<int32_t> bad = len;
            bad[0] = N + 1;
            CHECK(sekv::build_layout(&x, max_spans, ns.data(), bad.data(), off.data(), rk.data()) == -1);
            bad[0] = 0;
            CHECK(sekv::build_layout(&x, max_spans, ns.data(), bad.data(), off.data(), rk.data()) == -1);
        }
        std::vector<int32_t> many = ns;
        many[0] = max_spans + 1;
        CHECK(sekv::build_layout(&x, max_spans, many.data(), len.data(), off.data(), rk.data()) == -1);
        many[0] = -1;
        CHECK(sekv::build_layout(&x, max_spans, many.data(), len.data(), off.data(), rk.data()) == -1);
    }
    std::vector<int32_t> ns(3, 0), len(size_t(3) * d.max_tokens, 0);
    std::vector<int64_t> off(6);
    std::vector<int32_t> rk(6);
    CHECK(sekv::build_layout(&d, 1, ns.data(), len.data(), off.data(), rk.data()) == 256);
    CHECK(sekv::build_layout(&d, 0, ns.data(), len.data(), off.data(), rk.data()) == -1);
    CHECK(sekv::build_layout(&d, 1, nullptr, len.data(), off.data(), rk.data()) == -1);
    CHECK(sekv::build_layout(&d, 1, ns.data(), len.data(), nullptr, rk.data()) == -1);
}

}  // namespace

int main() {
    std::mt19937 rng(12345);
    test_check_dims();
    test_validate_cache(rng);
    test_tier_plan(rng);
    test_ws_tracker();
    test_build_layout(rng);
    if (g_fail) {
        std::printf("%d host checks failed\n", g_fail);
        return 1;
    }
    std::printf("all host checks passed\n");
    return 0;
}
