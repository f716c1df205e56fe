"""Pins of the oracle's prefill-side builder (Sec. 3.1 segmentation; Sec. 3.2 eq.
surprisal_weight summaries and eq. key_svd factors) to things other than itself: a
hand-worked example, library routines (numpy mean/std, math.fsum, numpy SVD), closed forms
and the invariants any segmentation under the rule has.  Planted mistakes must each break
at least one pin.  CPU only.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
import oracle.sekv_oracle as orc
from synth import make_prefill
from tests.helpers import rng

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "segmentation_worked_example.json")))


def check_worked_example():
    H = np.array(GOLD["H"], dtype=np.float32)
    mu, sigma, _ = orc.surprisal_threshold(H, H.size, 1.0)
    assert abs(mu - GOLD["mu"]) < GOLD["tolerance"] and abs(sigma - GOLD["sigma"]) < GOLD["tolerance"]
    for c in GOLD["cases"]:
        anchors, spans = orc.segment(H, H.size, c["alpha"], c["min_span"], c["window"])
        assert anchors == c["anchors"], c
        assert [list(s) for s in spans] == c["spans"], c


def check_stats_against_library():
    g = rng(5)
    for n in (1, 7, 1023, 1025, 5000):
        H = g.gamma(2.0, 1.0, n).astype(np.float32)
        mu, sigma, thr = orc.surprisal_threshold(H, n, 1.5)
        h = H.astype(np.float64)
        assert abs(mu - math.fsum(h) / n) <= 1e-13 * abs(mu)
        assert abs(sigma - np.std(h)) <= 1e-12 * max(np.std(h), 1e-300)
        assert thr == mu + 1.5 * sigma
    # the fixed order is exact where every partial sum is
    ints = np.arange(3000, dtype=np.float32) % 7
    assert orc._fixed_order_sum(ints.astype(np.float64)) == float(ints.sum())


def _check_partition(H, n, alpha, min_span, window):
    anchors, spans = orc.segment(H, n, alpha, min_span, window)
    _, _, thr = orc.surprisal_threshold(H, n, alpha)
    h = np.asarray(H, dtype=np.float32)[:n].astype(np.float64)
    cover = np.zeros(n, dtype=np.int32)
    cover[anchors] += 1
    for s, L in spans:
        assert L >= min_span
        cover[s:s + L] += 1
        # neighbours of a span are anchors or the sequence ends (maximal runs)
        assert s == 0 or cover[s - 1] >= 0 and (s - 1) in set(anchors)
        assert s + L == n or (s + L) in set(anchors)
    assert np.all(cover == 1), "anchors and spans must partition the tokens"
    assert set(np.flatnonzero(h > thr)) <= set(anchors)
    assert set(range(max(0, n - window), n)) <= set(anchors)
    assert all(a < b for a, b in zip(anchors, anchors[1:]))
    assert all(s0 + l0 <= s1 for (s0, l0), (s1, _) in zip(spans, spans[1:]))
    return anchors, spans


def check_segmentation_invariants():
    p = make_prefill(2, 1, 32, [3000, 2500], dtype="f32", seed=7)
    for b in range(2):
        n = int(p.n_tokens[b])
        for alpha, ms, w in ((1.0, 16, 512), (0.5, 4, 0), (2.0, 32, 100)):
            _check_partition(p.surprisal[b], n, alpha, ms, w)
    g = rng(8)
    H = g.exponential(1.0, 777).astype(np.float32)
    _check_partition(H, 777, 1.0, 3, 10)
    # no boundary at all (constant surprisal): one span before the window
    anchors, spans = orc.segment(np.ones(100, np.float32), 100, 1.0, 16, 20)
    assert anchors == list(range(80, 100)) and spans == [(0, 80)]


def check_weighted_summary():
    g = rng(9)
    X = g.standard_normal((13, 6))
    assert np.allclose(orc.weighted_summary(X, np.full(13, 3.0)), X.mean(axis=0), rtol=0, atol=1e-14)
    two = orc.weighted_summary(np.array([[1.0, 0.0], [0.0, 1.0]]), [3.0, 1.0])
    assert np.allclose(two, [0.75, 0.25], rtol=0, atol=1e-15)
    assert np.allclose(orc.weighted_summary(X, np.zeros(13)), X.mean(axis=0), rtol=0, atol=1e-14)


def check_truncated_svd():
    g = rng(10)
    for L, d, R in ((40, 16, 8), (5, 16, 8), (30, 8, 32)):
        X = g.standard_normal((L, d))
        U, s, Vt = orc.truncated_svd(X, R)
        r = min(L, d, R)
        assert U.shape == (L, r) and s.shape == (r,) and Vt.shape == (r, d)
        full = np.linalg.svd(X, compute_uv=False)
        err = np.linalg.norm(X - U @ np.diag(s) @ Vt) ** 2
        assert abs(err - np.sum(full[r:] ** 2)) <= 1e-10 * np.sum(full ** 2)
        assert np.allclose(U.T @ U, np.eye(r), atol=1e-12) and np.allclose(Vt @ Vt.T, np.eye(r), atol=1e-12)


def _dense_attention(q, K, V, n, scale):
    """Plain softmax attention of every query head over the first n tokens."""
    Hq, Hkv = q.shape[0], K.shape[0]
    G = Hq // Hkv
    out = np.zeros((Hq, K.shape[-1]))
    for h in range(Hq):
        s = K[h // G, :n] @ q[h] * scale
        w = np.exp(s - s.max())
        out[h] = (w / w.sum()) @ V[h // G, :n]
    return out


def _built(p, alpha, min_span, window, r_max, dtype):
    return orc.build_layer_cache(p.keys, p.values, p.surprisal, p.n_tokens, alpha=alpha,
                                 min_span=min_span, window=window, r_max=r_max, dtype=dtype)


def _decode(c, q, r_max, top_k, dtype):
    return orc.decode_step(q, c["anchor_k"], c["anchor_v"], c["n_anchors"], c["sum_k"], c["sum_v"],
                           c["n_spans"], c["span_len"], c["span_logsize"], c["factors"],
                           c["block_off"], rank=r_max, top_k=top_k, softmax_scale=0.25,
                           dtype=dtype, block_rank=c["block_rank"])


def check_built_cache_full_zoom_is_dense_attention():
    """Every span zoomed at full rank (r_max >= d): the built cache reproduces dense attention."""
    p = make_prefill(2, 2, 16, [90, 61], dtype="f32", spike_every=12, true_rank=6, seed=21)
    g = rng(22)
    q = g.standard_normal((2, 4, 16)).astype(np.float32)
    c = _built(p, 0.5, 3, 5, 16, "f32")
    assert int(c["n_spans"].min()) >= 2, "the pin needs spans"
    res = _decode(c, q, 16, int(c["n_spans"].max()), "f32")
    for b in range(2):
        n = int(p.n_tokens[b])
        ref = _dense_attention(q[b].astype(np.float64), p.keys[b].astype(np.float64),
                               p.values[b].astype(np.float64), n, 0.25)
        assert np.allclose(res["out"][b], ref, rtol=0, atol=2e-6), np.abs(res["out"][b] - ref).max()


def check_built_cache_constant_spans_unzoomed_is_dense_attention():
    """Tokens constant within each span: the coarse entries (summary logit + ln|S|, summary
    value) equal attention over the span's tokens, so no zoom at all gives dense attention."""
    p = make_prefill(1, 2, 16, [120], dtype="f32", spike_every=15, seed=23)
    anchors, spans = orc.segment(p.surprisal[0], 120, 1.0, 4, 7)
    assert len(spans) >= 2
    for s0, L in spans:
        p.keys[0, :, s0:s0 + L] = p.keys[0, :, s0:s0 + 1]
        p.values[0, :, s0:s0 + L] = p.values[0, :, s0:s0 + 1]
    q = rng(24).standard_normal((1, 4, 16)).astype(np.float32)
    c = _built(p, 1.0, 4, 7, 8, "f32")
    res = _decode(c, q, 8, 0, "f32")
    ref = _dense_attention(q[0].astype(np.float64), p.keys[0].astype(np.float64),
                           p.values[0].astype(np.float64), 120, 0.25)
    assert np.allclose(res["out"][0], ref, rtol=0, atol=1e-6), np.abs(res["out"][0] - ref).max()


def check_built_cache_layout():
    """Stored ranks round min(|S|, d, R_max) up to the granule; blocks hold the truncated SVD
    with zero extra components; anchors are the token rows; ln|S| natural."""
    p = make_prefill(1, 1, 32, [700], dtype="bf16", spike_every=60, seed=25)
    c = _built(p, 1.0, 2, 16, 24, "bf16")
    anchors, spans = c["segments"][0]
    assert np.array_equal(c["anchor_k"][0, 0, :len(anchors)], p.keys[0, 0, anchors])
    for S, (s0, L) in enumerate(spans):
        rk, rv = c["block_rank"][0, 0, S] & 0xFFFF, c["block_rank"][0, 0, S] >> 16
        r = min(L, 32, 24)
        assert rk == rv == -(-r // 8) * 8 and c["block_off"][0, 0, S] % 256 == 0
        assert c["span_len"][0, S] == L and c["span_logsize"][0, S] == math.log(L)
        blk = orc.read_span_block(c["factors"], int(c["block_off"][0, 0, S]), L, rk, 32, "bf16", rv)
        X = orc.widen(p.keys[0, 0, s0:s0 + L], "bf16")
        assert np.all(blk["sK"][r:] == 0) and np.all(blk["UK"][:, r:] == 0)
        full = np.linalg.svd(X, compute_uv=False)
        err = np.linalg.norm(X - orc.reconstruct(blk["UK"], blk["sK"], blk["VtK"]))
        assert err <= math.sqrt(np.sum(full[r:] ** 2)) + 2e-2 * np.linalg.norm(X)


PINS = [check_worked_example, check_stats_against_library, check_segmentation_invariants,
        check_weighted_summary, check_truncated_svd, check_built_cache_full_zoom_is_dense_attention,
        check_built_cache_constant_spans_unzoomed_is_dense_attention, check_built_cache_layout]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_build_pin(pin):
    pin()


_orig_seg = orc.segment
_orig_thr = orc.surprisal_threshold
_orig_ws = orc.weighted_summary
_orig_svd = orc.truncated_svd


def _no_alpha(H, n, alpha, *a):
    return _orig_seg(H, n, 1.0, *a)


def _sample_std(H, n, alpha):
    h = np.asarray(H, dtype=np.float32)[:n].astype(np.float64)
    mu = h.mean()
    sigma = float(np.std(h, ddof=1)) if n > 1 else 0.0
    return mu, sigma, mu + alpha * sigma


def _short_runs_kept(H, n, alpha, min_span, window):
    return _orig_seg(H, n, alpha, 1, window)


def _no_window(H, n, alpha, min_span, window):
    return _orig_seg(H, n, alpha, min_span, 0)


def _unnormalised(X, H):
    return np.asarray(H, dtype=np.float64) @ np.asarray(X, dtype=np.float64)


def _rank_off_by_one(X, r_max):
    U, s, Vt = _orig_svd(X, r_max)
    return U[:, :-1], s[:-1], Vt[:-1]


MUTANTS = {
    "alpha ignored": ("segment", _no_alpha),
    "sample standard deviation": ("surprisal_threshold", _sample_std),
    "short runs kept as spans": ("segment", _short_runs_kept),
    "no local window": ("segment", _no_window),
    "weights not normalised": ("weighted_summary", _unnormalised),
    "one component short": ("truncated_svd", _rank_off_by_one),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_build_planted_mistake_breaks_a_pin(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(orc, attr, fn)
    monkeypatch.setattr(oracle, attr, fn, raising=False)
    failed = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake: {name}"
