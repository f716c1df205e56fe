"""Pins of the CPU oracle to things other than itself.

Each check ties one step of the oracle to a library routine, a closed form, an
identity the paper states, or brute force on tiny inputs.  The mutation test at
the bottom plants plausible mistakes in the oracle and confirms that at least
one pin fails for each.  Everything here runs on the CPU.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import oracle.sekv_oracle as orc
from synth import case_from_factors, custom_spec, make_case
from synth.cases import bf16_bits_to_f64, from_storage
from tests.helpers import oracle_kwargs, rng


# ---------------------------------------------------------------------------
# builders
# ---------------------------------------------------------------------------

def _svd_factors(M, r):
    """Exact factors of M padded to rank r (zero components past rank)."""
    U, s, Vt = np.linalg.svd(M, full_matrices=False)
    k = s.size
    Up = np.zeros((M.shape[0], r)); Up[:, :k] = U
    sp = np.zeros(r); sp[:k] = s
    Vp = np.zeros((r, M.shape[1])); Vp[:k] = Vt
    return Up, sp, Vp


def _full_rank_cache(seed=0, dtype="f32", r=8, d=16, Hq=4, Hkv=2,
                     anchors=(5, 3), span_lens=((4, 6, 8), (5, 7)), top_k=8):
    """Cache whose spans are exact (full-rank) SVDs of known K/V matrices."""
    g = rng(seed)
    B = len(anchors)
    q = g.standard_normal((B, Hq, d))
    ak = [g.standard_normal((Hkv, A, d)) for A in anchors]
    av = [g.standard_normal((Hkv, A, d)) for A in anchors]
    originals = []
    spans = []
    for b in range(B):
        per_b, orig_b = [], []
        for L in span_lens[b]:
            heads, orig_h = [], []
            for _ in range(Hkv):
                K = g.standard_normal((L, d)); V = g.standard_normal((L, d))
                UK, sK, VtK = _svd_factors(K, r)
                UV, sV, VtV = _svd_factors(V, r)
                heads.append(dict(UK=UK, sK=sK, VtK=VtK, UV=UV, sV=sV, VtV=VtV))
                orig_h.append((K, V))
            per_b.append(heads); orig_b.append(orig_h)
        spans.append(per_b); originals.append(orig_b)
    case = case_from_factors(q, ak, av, spans, dtype=dtype, top_k=top_k)
    return case, originals


def _stored_recon(case, b, g, S, side):
    """Token matrix of a stored span, read straight from the arena by the test."""
    s = case.spec
    e = 4 if s.dtype == "f32" else 2
    L, r, d = int(case.span_len[b, S]), s.rank, s.head_dim
    base = int(case.block_off[b, g, S]) // e
    arr = case.factors.view(np.float32 if s.dtype == "f32" else np.uint16)
    seg = L * r + r + r * d
    o = base + (0 if side == "K" else seg)
    U = from_storage(arr[o:o + L * r], s.dtype).reshape(L, r)
    sig = from_storage(arr[o + L * r:o + L * r + r], s.dtype)
    Vt = from_storage(arr[o + L * r + r:o + seg], s.dtype).reshape(r, d)
    return np.einsum("tr,r,rd->td", U, sig, Vt)


def _sdpa(q, K, V, scale, bias=None):
    """torch's scaled-dot-product attention in float64 on the CPU, one query row."""
    qt = torch.tensor(q, dtype=torch.float64).reshape(1, 1, 1, -1)
    Kt = torch.tensor(K, dtype=torch.float64).reshape(1, 1, K.shape[0], -1)
    Vt = torch.tensor(V, dtype=torch.float64).reshape(1, 1, V.shape[0], -1)
    mask = None if bias is None else torch.tensor(bias, dtype=torch.float64).reshape(1, 1, 1, -1)
    out = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, attn_mask=mask, scale=scale)
    return out.reshape(-1).numpy()


# ---------------------------------------------------------------------------
# P1  full-rank factors reproduce the matrix (eq. key_svd / key_reconstruction)
# ---------------------------------------------------------------------------

def check_p1():
    g = rng(1)
    for L, d in [(5, 16), (16, 16), (12, 64), (3, 128)]:
        K = g.standard_normal((L, d))
        U, s, Vt = np.linalg.svd(K, full_matrices=False)
        assert np.max(np.abs(oracle.reconstruct(U, s, Vt) - K)) < 1e-12
    u, v = g.standard_normal(7), g.standard_normal(9)
    R1 = oracle.reconstruct(u[:, None], np.array([2.5]), v[None, :])
    assert np.max(np.abs(R1 - 2.5 * np.outer(u, v))) < 1e-13
    # through the stored block layout: parse + reconstruct matches the original K/V
    case, orig = _full_rank_cache(seed=2, dtype="f32")
    s = case.spec
    for b in range(case.spec.batch):
        for S in range(int(case.n_spans[b])):
            for gg in range(s.n_kv_heads):
                f = oracle.read_span_block(case.factors, int(case.block_off[b, gg, S]),
                                           int(case.span_len[b, S]), s.rank, s.head_dim, s.dtype)
                K, V = orig[b][S][gg]
                assert np.max(np.abs(oracle.reconstruct(f["UK"], f["sK"], f["VtK"]) - K)) < 1e-5
                assert np.max(np.abs(oracle.reconstruct(f["UV"], f["sV"], f["VtV"]) - V)) < 1e-5


def test_p1_full_rank_reconstruction():
    check_p1()


# ---------------------------------------------------------------------------
# P2  k = all spans equals dense attention over anchors + every reconstructed token
# ---------------------------------------------------------------------------

def check_p2():
    for dtype in ("f32", "bf16"):
        case, orig = _full_rank_cache(seed=3, dtype=dtype, top_k=8)
        s = case.spec
        res = oracle.decode_step(**oracle_kwargs(case))
        qd = from_storage(case.q, dtype)
        G = s.group
        for b in range(s.batch):
            m, A = int(case.n_spans[b]), int(case.n_anchors[b])
            for gg in range(s.n_kv_heads):
                assert sorted(res["sel"][b, gg, :m].tolist()) == list(range(m))
                assert np.all(res["sel"][b, gg, m:] == -1)
                Ks = [from_storage(case.anchor_k[b, gg, :A], dtype)]
                Vs = [from_storage(case.anchor_v[b, gg, :A], dtype)]
                Ko = [Ks[0]]; Vo = [Vs[0]]
                for S in range(m):
                    Ks.append(_stored_recon(case, b, gg, S, "K"))
                    Vs.append(_stored_recon(case, b, gg, S, "V"))
                    Ko.append(orig[b][S][gg][0]); Vo.append(orig[b][S][gg][1])
                K, V = np.concatenate(Ks), np.concatenate(Vs)
                for h in range(gg * G, (gg + 1) * G):
                    ref = _sdpa(qd[b, h], K, V, s.softmax_scale)
                    assert np.max(np.abs(res["out"][b, h] - ref)) < 1e-12
                    if dtype == "f32":
                        ref_o = _sdpa(qd[b, h], np.concatenate(Ko), np.concatenate(Vo),
                                      s.softmax_scale)
                        assert np.max(np.abs(res["out"][b, h] - ref_o)) < 2e-5


def test_p2_all_spans_equals_dense_attention():
    check_p2()


# ---------------------------------------------------------------------------
# P3  the weights of the one softmax sum to one
# ---------------------------------------------------------------------------

def check_p3():
    g = rng(4)
    d = 8
    ak, av = g.standard_normal((5, d)), g.standard_normal((5, d))
    cl, cv = g.standard_normal(3) * 30, g.standard_normal((3, d))
    zoom = [(g.standard_normal((4, d)), g.standard_normal((4, d)))]
    out, p = oracle.mixed_attention_head(g.standard_normal(d), 0.3, ak, av, cl, cv, zoom)
    assert p.shape == (5 + 3 + 4,)
    assert np.all(p >= 0) and abs(p.sum() - 1.0) < 1e-12
    assert np.allclose(out, p @ np.concatenate([av, cv, zoom[0][1]]), atol=1e-12, rtol=0)


def test_p3_softmax_weights_sum_to_one():
    check_p3()
    # and inside full decode steps (the oracle asserts it for every head)
    for variant in "LN":
        case = make_case(custom_spec(dtype="bf16", head_dim=64, rank=8, top_k=3), variant=variant)
        oracle.decode_step(**oracle_kwargs(case))


# ---------------------------------------------------------------------------
# P4  k = 0 equals attention over anchors + summaries with a ln|S| bias
# ---------------------------------------------------------------------------

def check_p4():
    for dtype, seed in (("f32", 5), ("bf16", 6)):
        spec = custom_spec(dtype=dtype, batch=2, n_q_heads=6, n_kv_heads=2, head_dim=32,
                           rank=8, top_k=0, context=400, seed=seed)
        case = make_case(spec)
        res = oracle.decode_step(**oracle_kwargs(case))
        assert res["sel"].shape == (2, 2, 0)
        qd = from_storage(case.q, dtype)
        for b in range(2):
            m, A = int(case.n_spans[b]), int(case.n_anchors[b])
            for h in range(6):
                gg = h // 3
                K = np.concatenate([from_storage(case.anchor_k[b, gg, :A], dtype),
                                    from_storage(case.sum_k[b, gg, :m], dtype)])
                V = np.concatenate([from_storage(case.anchor_v[b, gg, :A], dtype),
                                    from_storage(case.sum_v[b, gg, :m], dtype)])
                bias = np.concatenate([np.zeros(A), np.log(case.span_len[b, :m].astype(float))])
                ref = _sdpa(qd[b, h], K, V, spec.softmax_scale, bias)
                assert np.max(np.abs(res["out"][b, h] - ref)) < 1e-12


def test_p4_no_zoom_is_biased_attention_over_summaries():
    check_p4()


# ---------------------------------------------------------------------------
# P5  one coarse entry with +ln|S| weighs exactly like |S| identical tokens (Sec. 3.3)
# ---------------------------------------------------------------------------

def check_p5():
    g = rng(7)
    d, r, Hq, Hkv = 16, 8, 2, 1
    for L in (4, 16, 64):
        spans = []
        for j in range(3):
            Lj = L if j == 1 else 6
            if j == 1:   # identical rows: U = 1/sqrt(L), sigma = sqrt(L), v exact in fp32
                vk = np.round(g.standard_normal(d) * 8) / 8
                vv = np.round(g.standard_normal(d) * 8) / 8
                f = {}
                for side, v in (("K", vk), ("V", vv)):
                    U = np.zeros((Lj, r)); U[:, 0] = 1 / math.sqrt(Lj)
                    s = np.zeros(r); s[0] = math.sqrt(Lj)
                    Vt = np.zeros((r, d)); Vt[0] = v
                    f.update({"U" + side: U, "s" + side: s, "Vt" + side: Vt})
            else:
                f = {}
                for side in "KV":
                    f.update({"U" + side: g.standard_normal((Lj, r)),
                              "s" + side: np.abs(g.standard_normal(r)),
                              "Vt" + side: g.standard_normal((r, d))})
            spans.append([f])
        q = g.standard_normal((1, Hq, d))
        ak = [g.standard_normal((Hkv, 3, d))]
        case = case_from_factors(q, ak, [g.standard_normal((Hkv, 3, d))], [spans],
                                 dtype="f32", top_k=1)
        kw = oracle_kwargs(case)
        qd = from_storage(case.q, "f32")
        logits = orc.routing_logits(qd, from_storage(case.sum_k, "f32"), case.span_logsize,
                                    case.n_spans, case.spec.softmax_scale)
        common = {k: kw[k] for k in ("q", "anchor_k", "anchor_v", "n_anchors", "sum_v",
                                     "n_spans", "span_len", "factors", "block_off")}
        zoomed = oracle.zoom_attend(**common, sel=np.array([[[1]]], np.int32), logits=logits,
                                    rank=r, softmax_scale=case.spec.softmax_scale, dtype="f32")
        coarse = oracle.zoom_attend(**common, sel=np.array([[[-1]]], np.int32), logits=logits,
                                    rank=r, softmax_scale=case.spec.softmax_scale, dtype="f32")
        assert np.max(np.abs(zoomed - coarse)) < 1e-12


def test_p5_proportional_attention_identity():
    check_p5()


# ---------------------------------------------------------------------------
# P6  selection: brute-force rank counting, tie rule, padding
# ---------------------------------------------------------------------------

def _brute_select(keys_row, m, k):
    rank = [sum(1 for t in range(m) if (keys_row[t] > keys_row[S]) or
                (keys_row[t] == keys_row[S] and t < S)) for S in range(m)]
    out = [-1] * k
    for S in range(m):
        if rank[S] < k:
            out[rank[S]] = S
    return out


def check_p6():
    g = rng(8)
    B, Hkv, M = 3, 2, 40
    keys = np.round(g.standard_normal((B, Hkv, M)) * 3) / 3     # many exact ties
    n_spans = np.array([40, 17, 3])
    for k in (0, 1, 5, 17, 50):
        sel = oracle.select_topk(keys, n_spans, k)
        for b in range(B):
            for gg in range(Hkv):
                assert sel[b, gg].tolist() == _brute_select(keys[b, gg], int(n_spans[b]), k)
    # end to end: a duplicated span (same mean key, same length) ties; the lower index wins
    spec = custom_spec(dtype="bf16", n_q_heads=2, n_kv_heads=1, head_dim=32, rank=8, top_k=1,
                       context=300, seed=9)
    case = make_case(spec)
    res = oracle.decode_step(**oracle_kwargs(case))
    best = int(res["sel"][0, 0, 0])
    twin = best + 1 if best + 1 < int(case.n_spans[0]) else best - 1
    case.sum_k[0, 0, twin] = case.sum_k[0, 0, best]
    case.span_len[0, twin] = case.span_len[0, best]
    case.span_logsize[0, twin] = case.span_logsize[0, best]
    res2 = oracle.decode_step(**oracle_kwargs(case))
    assert res2["keys"][0, 0, twin] == res2["keys"][0, 0, best]
    assert int(res2["sel"][0, 0, 0]) == min(best, twin)


def test_p6_selection_brute_force_and_ties():
    check_p6()


# ---------------------------------------------------------------------------
# P7  coarse mean closed form; the generator's summaries are those means, rounded
# ---------------------------------------------------------------------------

def check_p7():
    g = rng(10)
    for L, r, d in [(7, 4, 16), (33, 8, 64)]:
        U, s, Vt = g.standard_normal((L, r)), np.abs(g.standard_normal(r)), g.standard_normal((r, d))
        closed = (U.sum(axis=0) / L * s) @ Vt
        mean = oracle.reconstruct(U, s, Vt).mean(axis=0)
        assert np.max(np.abs(closed - mean)) < 1e-13 * max(1.0, np.abs(mean).max())
    case = make_case(custom_spec(dtype="bf16", head_dim=64, rank=8, seed=11))
    sp = case.spec
    for S in range(int(case.n_spans[0])):
        for gg in range(sp.n_kv_heads):
            f = oracle.read_span_block(case.factors, int(case.block_off[0, gg, S]),
                                       int(case.span_len[0, S]), sp.rank, sp.head_dim, sp.dtype)
            for side, stored in (("K", case.sum_k), ("V", case.sum_v)):
                mean = oracle.reconstruct(f["U" + side], f["s" + side], f["Vt" + side]).mean(0)
                got = bf16_bits_to_f64(stored[0, gg, S])
                assert np.all(np.abs(got - mean) <= 2.0 ** -8 * np.abs(mean) + 1e-30)


def test_p7_summary_is_span_mean():
    check_p7()


# ---------------------------------------------------------------------------
# P8  factored attention identity (a second path to the zoomed scores/values)
# ---------------------------------------------------------------------------

def check_p8():
    g = rng(12)
    for L, r, d in [(9, 4, 16), (200, 32, 128)]:
        U, s, Vt = g.standard_normal((L, r)), np.abs(g.standard_normal(r)), g.standard_normal((r, d))
        qh = g.standard_normal(d)
        K_hat = oracle.reconstruct(U, s, Vt)
        a = oracle.zoom_scores_factored(qh, 0.125, U, s, Vt)
        assert np.max(np.abs(a - 0.125 * (K_hat @ qh))) < 1e-12 * max(1, np.abs(a).max())
        p = np.abs(g.standard_normal(L))
        V_hat = oracle.reconstruct(U, s, Vt)
        o = oracle.zoom_values_factored(p, U, s, Vt)
        assert np.max(np.abs(o - p @ V_hat)) < 1e-12 * max(1, np.abs(o).max())


def test_p8_factored_identity():
    check_p8()


# ---------------------------------------------------------------------------
# P9  GQA readings: G = 1 is per-head selection; max over the group; identical heads
# ---------------------------------------------------------------------------

def check_p9():
    # G = 1: a KV head's key is its one query head's score
    spec = custom_spec(dtype="f32", n_q_heads=3, n_kv_heads=3, head_dim=16, rank=4, top_k=3,
                       context=300, seed=13)
    case = make_case(spec)
    res = oracle.decode_step(**oracle_kwargs(case))
    assert np.array_equal(res["keys"], res["logits"])
    # max over the group: heads (a, b) and heads (a, b, b, b) select the same spans,
    # on summaries built so that group means would rank differently
    g = rng(14)
    d, r = 16, 4
    spans = [[{"UK": g.standard_normal((8, r)), "sK": np.ones(r), "VtK": g.standard_normal((r, d)),
               "UV": g.standard_normal((8, r)), "sV": np.ones(r), "VtV": g.standard_normal((r, d))}]
             for _ in range(4)]
    kbar = np.zeros((1, 1, 4, d))
    kbar[0, 0, :, :2] = [[3, 0], [0, 3], [2, 2], [2.25, 1.5]]
    a_vec, b_vec = np.eye(d)[0], np.eye(d)[1]
    anchors_k, anchors_v = [g.standard_normal((1, 2, d))], [g.standard_normal((1, 2, d))]
    c2 = case_from_factors(np.stack([a_vec, b_vec])[None], anchors_k, anchors_v, [spans],
                           dtype="f32", top_k=1, sum_k=kbar)
    c4 = case_from_factors(np.stack([a_vec, b_vec, b_vec, b_vec])[None], anchors_k, anchors_v,
                           [spans], dtype="f32", top_k=1, sum_k=kbar)
    r2 = oracle.decode_step(**oracle_kwargs(c2))
    r4 = oracle.decode_step(**oracle_kwargs(c4))
    assert r2["sel"].tolist() == r4["sel"].tolist() == [[[0]]]
    # identical heads give identical outputs
    assert np.array_equal(r4["out"][0, 1], r4["out"][0, 2])
    # the data separates the readings: group means would select differently
    mean2 = r2["logits"].reshape(1, 1, 2, -1).mean(axis=2)
    mean4 = r4["logits"].reshape(1, 1, 4, -1).mean(axis=2)
    assert oracle.select_topk(mean2, c2.n_spans, 1).tolist() == [[[2]]]
    assert oracle.select_topk(mean4, c4.n_spans, 1).tolist() == [[[1]]]


def test_p9_gqa_readings():
    check_p9()


# ---------------------------------------------------------------------------
# P10  split softmax: partials over any partition merge to the one softmax
# ---------------------------------------------------------------------------

def check_p10():
    g = rng(15)
    for n in (1, 7, 300):
        logits = g.standard_normal(n) * 10
        values = g.standard_normal((n, 5))
        ref = oracle.softmax_weights(logits) @ values
        for _ in range(5):
            cuts = np.sort(g.integers(0, n + 1, size=g.integers(0, 6)))
            bounds = [0, *cuts.tolist(), n]
            parts = [oracle.softmax_partial(logits[a:b], values[a:b])
                     for a, b in zip(bounds[:-1], bounds[1:])]
            assert np.max(np.abs(oracle.merge_partials(parts) - ref)) < 1e-12


def test_p10_split_softmax_merge():
    check_p10()


# ---------------------------------------------------------------------------
# P11  orthonormal factors: energy and truncation error (Sec. 3.3, reconstruction loss)
# ---------------------------------------------------------------------------

def check_p11():
    g = rng(16)
    L, r, d = 40, 8, 64
    U = np.linalg.qr(g.standard_normal((L, r)))[0]
    Vt = np.linalg.qr(g.standard_normal((d, r)))[0].T
    s = np.sort(np.abs(g.standard_normal(r)))[::-1] * 3
    K = oracle.reconstruct(U, s, Vt)
    assert abs(np.sum(K * K) - np.sum(s * s)) < 1e-12 * np.sum(s * s)
    for j in range(r + 1):
        Kj = oracle.reconstruct(U[:, :j], s[:j], Vt[:j])
        err = np.sum((K - Kj) ** 2)
        assert abs(err - np.sum(s[j:] ** 2)) < 1e-12 * np.sum(s * s)
    m = g.uniform(0, 1, r)            # soft rank gates folded into sigma
    err = np.sum((K - oracle.reconstruct(U, m * s, Vt)) ** 2)
    assert abs(err - np.sum((1 - m) ** 2 * s ** 2)) < 1e-12 * np.sum(s * s)


def test_p11_orthonormal_energy_and_truncation():
    check_p11()


# ---------------------------------------------------------------------------
# the routing score's float64 contract (left-to-right sum, then * scale, then + ln|S|)
# ---------------------------------------------------------------------------

def test_routing_score_bitwise_contract():
    case = make_case(custom_spec(dtype="bf16", n_q_heads=4, n_kv_heads=2, head_dim=32,
                                 rank=8, context=200, seed=17))
    qd, kd = from_storage(case.q, "bf16"), from_storage(case.sum_k, "bf16")
    lg = orc.routing_logits(qd, kd, case.span_logsize, case.n_spans, case.spec.softmax_scale)
    for h in range(4):
        for S in range(int(case.n_spans[0])):
            s = 0.0
            for j in range(32):
                s = s + float(qd[0, h, j]) * float(kd[0, h // 2, S, j])
            ref = s * case.spec.softmax_scale + float(case.span_logsize[0, S])
            assert lg[0, h, S] == ref
            exact = math.fsum(float(qd[0, h, j]) * float(kd[0, h // 2, S, j]) for j in range(32))
            assert abs(s - exact) <= 1e-15 * max(1e-300, sum(abs(float(qd[0, h, j]) *
                                                              float(kd[0, h // 2, S, j]))
                                                          for j in range(32)))


# ---------------------------------------------------------------------------
# planted mistakes: each must break at least one pin
# ---------------------------------------------------------------------------

PINS = [check_p1, check_p2, check_p4, check_p5, check_p6, check_p8, check_p9, check_p11]


def _drop_logsize(q, sum_k, span_logsize, n_spans, scale):
    return _orig_routing(q, sum_k, np.zeros_like(span_logsize), n_spans, scale)


def _log2_size(q, sum_k, span_logsize, n_spans, scale):
    return _orig_routing(q, sum_k, span_logsize / math.log(2), n_spans, scale)


def _scaled_logsize(q, sum_k, span_logsize, n_spans, scale):
    return _orig_routing(q, sum_k, span_logsize * scale, n_spans, scale)


def _no_sigma(U, sigma, Vt):
    return U @ Vt


def _transposed_sigma_use(U, sigma, Vt):
    return (U * sigma[::-1]) @ Vt


def _ties_high(keys, n_spans, k):
    B, Hkv, M = keys.shape
    sel = np.full((B, Hkv, k), -1, dtype=np.int32)
    for b in range(B):
        m = int(n_spans[b])
        for g in range(Hkv):
            order = sorted(range(m), key=lambda S: (-keys[b, g, S], -S))[:min(k, m)]
            sel[b, g, :len(order)] = order
    return sel


def _mean_group(logits, n_kv_heads):
    B, Hq, M = logits.shape
    return logits.reshape(B, n_kv_heads, Hq // n_kv_heads, M).mean(axis=2)


def _keep_coarse(q, anchor_k, anchor_v, n_anchors, sum_v, n_spans, span_len, factors,
                 block_off, sel, logits, *, rank, softmax_scale, dtype, block_rank=None):
    none = np.full_like(sel, -1)
    # coarse entries of every span stay, and the zoomed tokens are added on top
    qf = orc.widen(q, dtype)
    ak, av, sv = orc.widen(anchor_k, dtype), orc.widen(anchor_v, dtype), orc.widen(sum_v, dtype)
    B, Hq, d = qf.shape
    Hkv = ak.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, d))
    for b in range(B):
        A, m = int(n_anchors[b]), int(n_spans[b])
        for g in range(Hkv):
            zoom = []
            for S in [int(x) for x in sel[b, g] if x >= 0]:
                rk, rv = orc.block_ranks(block_rank, b, g, S, rank)
                f = orc.read_span_block(factors, int(block_off[b, g, S]), int(span_len[b, S]),
                                        rk, d, dtype, rank_v=rv)
                zoom.append((orc.reconstruct(f["UK"], f["sK"], f["VtK"]),
                             orc.reconstruct(f["UV"], f["sV"], f["VtV"])))
            for h in range(g * G, (g + 1) * G):
                out[b, h], _ = orc.mixed_attention_head(qf[b, h], softmax_scale, ak[b, g, :A],
                                                        av[b, g, :A], logits[b, h, :m],
                                                        sv[b, g, :m], zoom)
    del none
    return out


_orig_routing = orc.routing_logits

MUTANTS = {
    "routing drops ln|S|": ("routing_logits", _drop_logsize),
    "routing uses log2|S|": ("routing_logits", _log2_size),
    "routing scales ln|S|": ("routing_logits", _scaled_logsize),
    "reconstruction drops sigma": ("reconstruct", _no_sigma),
    "reconstruction misorders sigma": ("reconstruct", _transposed_sigma_use),
    "ties go to the higher index": ("select_topk", _ties_high),
    "group key is the mean": ("group_keys", _mean_group),
    "zoomed span keeps its coarse entry": ("zoom_attend", _keep_coarse),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_breaks_a_pin(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(orc, attr, fn)
    monkeypatch.setattr(oracle, attr, fn, raising=False)
    failed = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake: {name}"
