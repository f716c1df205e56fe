"""Pins of the oracle's learned selection rule to things other than itself.

The rule (Sec. 3.2 eqs. surprisal_weight, summary_key, query_projection,
routing_gate; Sec. 3.3 eq. zoom_decision and the budget cap) is checked
against a hand-worked example, closed forms, the identity-projection special
case (which must reduce to the top-k rule bit for bit), library routines, and
properties any correct selection has.  Planted mistakes at the bottom must each
break at least one pin.  CPU only.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
import oracle.sekv_oracle as orc
from synth import NO_BUDGET, custom_spec, make_case, make_gate
from synth.cases import from_storage
from tests.helpers import oracle_kwargs, rng

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "gated_worked_example.json")))


def _gated_kwargs(case, gate, max_zoom, budget):
    kw = oracle_kwargs(case)
    kw.pop("top_k")
    return dict(kw, proj=gate.proj, sum_route=gate.sum_route, thresholds=gate.thresholds,
                max_zoom=max_zoom, budget_tokens=budget)


def _case(seed=21, dtype="bf16", **kw):
    base = dict(dtype=dtype, n_q_heads=8, n_kv_heads=2, head_dim=32, rank=8, context=900,
                span_min=8, span_max=40, seed=seed)
    base.update(kw)
    return make_case(custom_spec(**base))


# ---------------------------------------------------------------------------
# the pins (check_* are reused by the planted-mistake test)
# ---------------------------------------------------------------------------

def check_worked_example():
    inp, exp = GOLD["inputs"], GOLD["expected"]
    tol = exp["tolerance"]
    q = np.array(inp["q"], dtype=np.float64)
    W = np.array(inp["proj"], dtype=np.float64)
    kr = np.array(inp["sum_route"], dtype=np.float64)
    span_len = np.array(inp["span_len"], dtype=np.int32)
    lns = np.log(span_len.astype(np.float64))
    n_spans = np.array([3], dtype=np.int32)
    qp = orc.project_queries(q, W)
    assert np.array_equal(qp, np.array(exp["q_proj"]))
    x = orc.gate_logits(qp, kr, lns, n_spans)
    assert np.allclose(x, np.array(exp["gate_logits"]), rtol=0, atol=tol)
    thr = orc.threshold_logit(np.array(inp["tau"]))
    assert np.allclose(thr, exp["thresholds"], rtol=0, atol=tol)
    assert abs(orc.gate(x)[0, 1, 1] - exp["alpha_head1_span1"]) < tol
    for case in exp["selections"]:
        sel = orc.gated_selection(x, thr, span_len, n_spans, 1, case["max_zoom"], case["budget_tokens"])
        assert sel[0, 0].tolist() == case["sel"], case


def check_identity_reduces_to_topk():
    """W = I, d' = d, the routing summary fed as the mean key, thresholds -inf, no
    budget: the gate is the identity routing score bit for bit, and the selection
    is the top-k rule."""
    case = _case(seed=22)
    s = case.spec
    G = s.n_q_heads // s.n_kv_heads
    d = s.head_dim
    qd = from_storage(case.q, s.dtype)
    kd = from_storage(case.sum_k, s.dtype)
    eye = np.broadcast_to(np.eye(d), (s.n_q_heads, d, d))
    qp = orc.project_queries(qd, eye)
    assert np.array_equal(qp, qd)
    kr = np.repeat(kd, G, axis=1)
    x = orc.gate_logits(qp, kr, case.span_logsize, case.n_spans)
    ref = orc.routing_logits(qd, kd, case.span_logsize, case.n_spans, s.softmax_scale)
    assert np.array_equal(x, ref)
    thr = np.full(s.n_q_heads, -np.inf)
    for k in (1, 3, 7):
        sel = orc.gated_selection(x, thr, case.span_len, case.n_spans, s.n_kv_heads, k, NO_BUDGET)
        top = orc.select_topk(orc.group_keys(ref, s.n_kv_heads), case.n_spans, k)
        assert np.array_equal(sel, top)


def check_summary_key():
    g = rng(3)
    K = g.standard_normal((11, 6))
    W = np.eye(6)
    w = orc.surprisal_weights(np.full(11, 2.5))
    assert np.allclose(w, 1.0 / 11, rtol=0, atol=1e-15)
    ks = orc.summary_key(K, w, W)
    mean = np.mean(K, axis=0)
    assert np.allclose(ks, mean / np.linalg.norm(mean), rtol=0, atol=1e-14)
    H = g.uniform(0.5, 4.0, 11)
    wt = orc.surprisal_weights(H)
    assert abs(wt.sum() - 1.0) < 1e-15 and np.all(wt > 0)
    Wr = g.standard_normal((3, 6))
    a = orc.summary_key(K, wt, Wr)
    assert abs(np.linalg.norm(a) - 1.0) < 1e-14
    perm = g.permutation(11)
    assert np.allclose(orc.summary_key(K[perm], wt[perm], Wr), a, rtol=0, atol=1e-14)
    assert np.allclose(orc.summary_key(3.0 * K, wt, Wr), a, rtol=0, atol=1e-14)
    # weight is proportional to surprisal: doubling one token's H moves the summary
    # towards that token's projected key (closed form for two tokens)
    K2 = np.array([[1.0, 0.0], [0.0, 1.0]])
    b = orc.summary_key(K2, orc.surprisal_weights([3.0, 1.0]), np.eye(2))
    assert np.allclose(b, np.array([3.0, 1.0]) / math.sqrt(10.0), rtol=0, atol=1e-15)


def check_projection_rounding():
    g = rng(4)
    q = g.standard_normal((2, 4, 16)).astype(np.float32).astype(np.float64)
    W = g.standard_normal((4, 5, 16)).astype(np.float32).astype(np.float64)
    qp = orc.project_queries(q, W)
    lib = np.einsum("hij,bhj->bhi", W, q)
    assert np.array_equal(qp, qp.astype(np.float32).astype(np.float64))
    ulp = np.spacing(np.abs(lib).astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(qp - lib) <= ulp)


def check_gate_dot_is_exact_sum():
    case = _case(seed=23, dtype="f32")
    gate = make_gate(case, route_dim=8, tau="spread")
    qd = from_storage(case.q, "f32")
    qp = orc.project_queries(qd, from_storage(gate.proj, "f32"))
    kr = from_storage(gate.sum_route, "f32")
    x = orc.gate_logits(qp, kr, case.span_logsize, case.n_spans)
    scale = 1.0 / math.sqrt(8.0)
    for h in (0, 5):
        for S in range(0, int(case.n_spans[0]), 7):
            prods = [float(qp[0, h, i]) * float(kr[0, h, S, i]) for i in range(8)]
            s = 0.0
            for p in prods:
                s = s + p
            assert abs(s - math.fsum(prods)) <= 1e-15 * sum(abs(p) for p in prods) + 1e-300
            assert x[0, h, S] == s * scale + float(case.span_logsize[0, S])
    assert np.all(np.isneginf(x[:, :, int(case.n_spans.max()):]))


def check_generator_summary_is_eq_summary_key():
    """The generator's routing summary equals eq. summary_key over the span's tokens
    (reconstructed from the stored factors, uniform weights), up to storage rounding."""
    for dt, tol in (("f32", 2e-6), ("bf16", 2e-2)):
        case = _case(seed=24, dtype=dt, n_q_heads=4, head_dim=16, context=300)
        gate = make_gate(case, route_dim=8)
        s = case.spec
        G = s.n_q_heads // s.n_kv_heads
        Wd = from_storage(gate.proj, dt)
        kr = from_storage(gate.sum_route, dt)
        for h in range(s.n_q_heads):
            for S in range(int(case.n_spans[0])):
                L = int(case.span_len[0, S])
                f = orc.read_span_block(case.factors, int(case.block_off[0, h // G, S]), L,
                                        s.rank, s.head_dim, dt)
                K = orc.reconstruct(f["UK"], f["sK"], f["VtK"])
                ref = orc.summary_key(K, orc.surprisal_weights(np.ones(L)), Wd[h])
                assert np.max(np.abs(kr[0, h, S] - ref)) < tol


def check_selection_properties():
    for seed, budget, k in ((25, 300, 6), (26, 120, 64), (27, NO_BUDGET, 5), (28, 0, 4)):
        case = _case(seed=seed)
        gate = make_gate(case, route_dim=16, tau="spread", budget_tokens=budget)
        s = case.spec
        G = s.n_q_heads // s.n_kv_heads
        r = orc.decode_step_gated(**_gated_kwargs(case, gate, k, budget))
        x, sel = r["gate_logits"], r["sel"]
        alpha = orc.gate(x)
        for b in range(s.batch):
            m = int(case.n_spans[b])
            for g in range(s.n_kv_heads):
                heads = list(range(g * G, (g + 1) * G))
                chosen = [int(S) for S in sel[b, g] if S >= 0]
                assert sel[b, g, len(chosen):].tolist() == [-1] * (k - len(chosen))
                assert len(set(chosen)) == len(chosen) <= k
                assert sum(int(case.span_len[b, S]) for S in chosen) <= budget
                # every expanded span has a head whose gate exceeds its tau (probability space)
                for S in chosen:
                    assert any(alpha[b, h, S] > gate.tau[h] for h in heads)
                voted = [S for S in range(m) if any(alpha[b, h, S] > gate.tau[h] for h in heads)]
                key = {S: max(x[b, h, S] for h in heads if alpha[b, h, S] > gate.tau[h]) for S in voted}
                # chosen are in expansion order and ahead of every voted span left out
                for a_, c_ in zip(chosen, chosen[1:]):
                    assert (key[a_], -a_) > (key[c_], -c_)
                rest = [S for S in voted if S not in chosen]
                for S in rest:
                    assert all((key[c], -c) > (key[S], -S) for c in chosen)
                # maximal: the best voted span left out would break the count or the budget
                if rest:
                    nxt = max(rest, key=lambda S: (key[S], -S))
                    used = sum(int(case.span_len[b, S]) for S in chosen)
                    assert len(chosen) == k or used + int(case.span_len[b, nxt]) > budget


def check_degenerate_rules():
    case = _case(seed=29)
    s = case.spec
    gate = make_gate(case, route_dim=16, tau="spread")
    kw = _gated_kwargs(case, gate, 5, NO_BUDGET)
    none = np.full((s.batch, s.n_kv_heads, 5), -1, dtype=np.int32)
    assert np.array_equal(orc.decode_step_gated(**dict(kw, budget_tokens=0))["sel"], none)
    assert np.array_equal(orc.decode_step_gated(**dict(kw, thresholds=np.full(s.n_q_heads, np.inf)))["sel"], none)
    r0 = orc.decode_step_gated(**dict(kw, max_zoom=0))
    assert r0["sel"].shape == (s.batch, s.n_kv_heads, 0)
    # nothing expanded: the output is attention over anchors and all coarse entries
    base = oracle_kwargs(case)
    ref = orc.zoom_attend(base["q"], base["anchor_k"], base["anchor_v"], base["n_anchors"],
                          base["sum_v"], base["n_spans"], base["span_len"], base["factors"],
                          base["block_off"], none,
                          orc.routing_logits(from_storage(case.q, s.dtype),
                                             from_storage(case.sum_k, s.dtype),
                                             case.span_logsize, case.n_spans, s.softmax_scale),
                          rank=s.rank, softmax_scale=s.softmax_scale, dtype=s.dtype)
    assert np.array_equal(orc.decode_step_gated(**dict(kw, budget_tokens=0))["out"], ref)
    # thresholds in logit space match tau in probability space
    taus = np.array([0.05, 0.3, 0.5, 0.9, 0.999])
    assert np.allclose(orc.gate(orc.threshold_logit(taus)), taus, rtol=1e-14, atol=0)
    assert np.allclose(orc.threshold_logit(gate.tau), gate.thresholds, rtol=1e-13, atol=1e-15)


def check_identity_step_equals_topk_step():
    """The full step under the identity reading of the gate equals the top-k step."""
    case = _case(seed=30, dtype="f32", n_q_heads=4, head_dim=16, context=400)
    s = case.spec
    G = s.n_q_heads // s.n_kv_heads
    d = s.head_dim
    ident = make_gate(case, route_dim=d, proj_f64=np.broadcast_to(np.eye(d), (s.n_q_heads, d, d)))
    ident.sum_route = np.repeat(case.sum_k, G, axis=1)
    kw = _gated_kwargs(case, ident, s.top_k, NO_BUDGET)
    kw["thresholds"] = np.full(s.n_q_heads, -np.inf)
    r = orc.decode_step_gated(**kw)
    ref = orc.decode_step(**oracle_kwargs(case))
    assert np.array_equal(r["sel"], ref["sel"])
    assert np.array_equal(r["out"], ref["out"])


PINS = [check_worked_example, check_identity_reduces_to_topk, check_summary_key,
        check_projection_rounding, check_gate_dot_is_exact_sum,
        check_generator_summary_is_eq_summary_key, check_selection_properties,
        check_degenerate_rules, check_identity_step_equals_topk_step]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_gated_pin(pin):
    pin()


# ---------------------------------------------------------------------------
# planted mistakes: each must break at least one pin
# ---------------------------------------------------------------------------

_orig_gate_logits = orc.gate_logits
_orig_selection = orc.gated_selection
_orig_project = orc.project_queries


def _scale_by_d(q_proj, sum_route, span_logsize, n_spans):
    x = _orig_gate_logits(q_proj, sum_route, span_logsize, n_spans)
    dr = np.asarray(q_proj).shape[2]
    return (x - np.asarray(span_logsize)[:, None, :x.shape[2]]) / math.sqrt(dr) * math.sqrt(dr) * 0.5 + \
        np.asarray(span_logsize)[:, None, :x.shape[2]]


def _no_logsize(q_proj, sum_route, span_logsize, n_spans):
    return _orig_gate_logits(q_proj, sum_route, np.zeros_like(span_logsize), n_spans)


def _no_round(q, W):
    q = np.asarray(q, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    return np.einsum("hij,bhj->bhi", W, q) * (1.0 + 1e-9)


def _transposed_proj(q, W):
    return _orig_project(q, np.swapaxes(np.asarray(W), 1, 2)[:, :np.asarray(W).shape[1], :]
                         if np.asarray(W).shape[1] == np.asarray(W).shape[2] else W[:, ::-1, :])


def _skip_instead_of_stop(x, thresholds, span_len, n_spans, n_kv_heads, max_zoom, budget_tokens):
    B, Hq, M = x.shape
    G = Hq // n_kv_heads
    sel = np.full((B, n_kv_heads, max_zoom), -1, dtype=np.int32)
    for b in range(B):
        for g in range(n_kv_heads):
            hs = range(g * G, (g + 1) * G)
            c = sorted(((max(x[b, h, S] for h in hs if x[b, h, S] > thresholds[h]), S)
                        for S in range(int(n_spans[b])) if any(x[b, h, S] > thresholds[h] for h in hs)),
                       key=lambda t: (-t[0], t[1]))
            used, ch = 0, []
            for _, S in c:
                if len(ch) < max_zoom and used + int(span_len[b, S]) <= budget_tokens:
                    ch.append(S)
                    used += int(span_len[b, S])
            sel[b, g, :len(ch)] = ch
    return sel


def _one_threshold(x, thresholds, *a):
    return _orig_selection(x, np.full_like(np.asarray(thresholds, np.float64), thresholds[0]), *a)


def _key_from_all_heads(x, thresholds, span_len, n_spans, n_kv_heads, max_zoom, budget_tokens):
    B, Hq, M = x.shape
    G = Hq // n_kv_heads
    sel = np.full((B, n_kv_heads, max_zoom), -1, dtype=np.int32)
    for b in range(B):
        for g in range(n_kv_heads):
            hs = range(g * G, (g + 1) * G)
            c = sorted(((min(x[b, h, S] for h in hs), S) for S in range(int(n_spans[b]))
                        if any(x[b, h, S] > thresholds[h] for h in hs)), key=lambda t: (-t[0], t[1]))
            used, ch = 0, []
            for _, S in c:
                if len(ch) == max_zoom or used + int(span_len[b, S]) > budget_tokens:
                    break
                ch.append(S)
                used += int(span_len[b, S])
            sel[b, g, :len(ch)] = ch
    return sel


def _reversed_order(x, thresholds, span_len, n_spans, n_kv_heads, max_zoom, budget_tokens):
    return _orig_selection(np.round(x, 1), thresholds, span_len, n_spans, n_kv_heads, max_zoom,
                           budget_tokens)[..., ::-1].copy()


MUTANTS = {
    "gate scaled by 1/(2 sqrt d')": ("gate_logits", _scale_by_d),
    "gate drops ln|S|": ("gate_logits", _no_logsize),
    "projection not rounded to float32": ("project_queries", _no_round),
    "projection transposed": ("project_queries", _transposed_proj),
    "budget skips instead of stopping": ("gated_selection", _skip_instead_of_stop),
    "one threshold for every head": ("gated_selection", _one_threshold),
    "order key over all heads (min)": ("gated_selection", _key_from_all_heads),
    "selection order reversed": ("gated_selection", _reversed_order),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_gated_planted_mistake_breaks_a_pin(name, monkeypatch):
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
