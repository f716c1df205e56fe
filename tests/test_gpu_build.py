"""GPU parity of the prefill-side builder (Sec. 3.1 segmentation; Sec. 3.2 eq.
surprisal_weight summaries and eq. key_svd factors) against the CPU oracle.

* Segmentation: anchors and spans bit for bit (ragged batches, empty and one-token
  sequences, zero variance, window longer than the sequence, every token a boundary, the
  128K x 4 workload at full size).
* Anchor rows and span lengths bit for bit; ln|S| within 2 ulp; summaries within one
  storage ulp plus the float32 accumulation bound 1e-4 max|X|.
* Factors: the GPU's randomized SVD against the optimal truncated SVD (numpy): Frobenius
  reconstruction error at most 1.25 x the optimal with one or more subspace iterations
  (2 x with none) plus the storage rounding term (2^-7 ||X|| for bfloat16, 1e-5 ||X|| for
  float32); orthonormal columns of U and rows of Vt; stored ranks and zero extra
  components.
* End to end: the decode step on the GPU-built cache against the oracle's decode step on
  the oracle-built cache (exact SVD) for exactly low-rank spans, where both
  factorisations reproduce the span: selection equal wherever the oracle's k-th and
  (k+1)-th keys are apart, outputs within the decode step's tolerances.
"""

import math

import numpy as np
import pytest

import oracle
from synth import make_prefill
from tests.gpu_common import assert_out_close, banner, out_to_f64
from tests.helpers import rng

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


def _dev(a, dtype=None):
    import torch
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def _bdims(S, p, Hkv, d, rank=32, sketch=40, alpha=1.0, min_span=16, window=64, sweeps=8, power=1):
    return S.make_build_dims(batch=p.surprisal.shape[0], n_kv_heads=Hkv, head_dim=d,
                             max_tokens=p.surprisal.shape[1], rank=rank, sketch=sketch,
                             min_span=min_span, window=window, dtype=p.dtype, alpha=alpha,
                             sweeps=sweeps, power=power)


def _segment(S, bd, p):
    import torch
    seg = S.segment(bd, _dev(p.surprisal), _dev(p.n_tokens))
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in seg.items() if not k.startswith("_")}


def _check_segments(got, p, alpha, min_span, window, where):
    for b in range(p.surprisal.shape[0]):
        anchors, spans = oracle.segment(p.surprisal[b], int(p.n_tokens[b]), alpha, min_span, window)
        na, ns = int(got["n_anchors"][b]), int(got["n_spans"][b])
        assert na == len(anchors) and ns == len(spans), (where, b, na, len(anchors), ns, len(spans))
        assert got["anchor_idx"][b, :na].tolist() == anchors, (where, b)
        assert list(zip(got["span_start"][b, :ns].tolist(), got["span_len"][b, :ns].tolist())) == spans, \
            (where, b)


SEG_CASES = [
    ("ragged", dict(n=[3000, 1, 0, 2047], alpha=1.0, min_span=16, window=512, spike=150)),
    ("short-runs", dict(n=[4000, 999], alpha=0.5, min_span=2, window=0, spike=40)),
    ("negative-alpha", dict(n=[1500], alpha=-0.5, min_span=3, window=10, spike=150)),
    ("large-alpha", dict(n=[2500, 70], alpha=40.0, min_span=8, window=30, spike=150)),
    ("window-covers", dict(n=[300, 5], alpha=1.0, min_span=4, window=1000, spike=30)),
    ("min-span-too-long", dict(n=[600], alpha=1.0, min_span=601, window=0, spike=60)),
]


@pytest.mark.parametrize("name,c", SEG_CASES, ids=[c[0] for c in SEG_CASES])
def test_segment_matches_oracle(S, name, c):
    banner(f"segment {name}")
    p = make_prefill(len(c["n"]), 1, 64, c["n"], dtype="f32", spike_every=c["spike"], seed=71)
    bd = _bdims(S, p, 1, 64, alpha=c["alpha"], min_span=c["min_span"], window=c["window"])
    _check_segments(_segment(S, bd, p), p, c["alpha"], c["min_span"], c["window"], name)


def test_segment_zero_variance(S):
    banner("segment zero variance")
    p = make_prefill(2, 1, 64, [5000, 1024], dtype="f32", seed=72)
    p.surprisal[:] = 1.0
    bd = _bdims(S, p, 1, 64, window=100)
    got = _segment(S, bd, p)
    _check_segments(got, p, 1.0, 16, 100, "zero variance")
    assert got["n_spans"].tolist() == [1, 1]


def test_segment_full_size_128k_x4(S):
    banner("segment 131072 x 4")
    p = make_prefill(4, 1, 64, 131072, dtype="bf16", spike_every=170, true_rank=2, seed=73)
    bd = _bdims(S, p, 1, 64, min_span=16, window=512)
    _check_segments(_segment(S, bd, p), p, 1.0, 16, 512, "128k")


BUILD_CASES = [
    ("bf16-d128", dict(dtype="bf16", d=128, Hkv=2, n=[1500, 900], rank=32, sketch=40, min_span=4, window=64)),
    ("f32-d64", dict(dtype="f32", d=64, Hkv=2, n=[1200, 1], rank=32, sketch=40, min_span=2, window=16)),
    ("bf16-d64-r40-p2", dict(dtype="bf16", d=64, Hkv=1, n=[2000], rank=40, sketch=40, min_span=8, window=0,
                             power=2)),
    ("f32-d128-r8", dict(dtype="f32", d=128, Hkv=3, n=[800, 1100, 0], rank=8, sketch=12, min_span=3,
                         window=32)),
    # no subspace iteration: a plain Gaussian sketch, whose error bound is looser
    ("bf16-d128-p0", dict(dtype="bf16", d=128, Hkv=1, n=[1800], rank=16, sketch=24, min_span=4, window=16,
                          power=0, bound=2.0)),
]


def _build(S, p, c, ws_dims=None):
    import torch
    bd = _bdims(S, p, c["Hkv"], c["d"], rank=c["rank"], sketch=c["sketch"], min_span=c["min_span"],
                window=c["window"], power=c.get("power", 1))
    # the builder uses only the workspace's error word: any valid dims will do
    dims = S.make_dims(batch=1, n_q_heads=1, n_kv_heads=1, head_dim=64, rank=8, top_k=1, max_anchors=1,
                       max_spans=1, max_span_len=1, dtype="f32", softmax_scale=1.0)
    ws = S.Workspace(dims)
    cache, seg, lay = S.build_layer(bd, _dev(p.keys, p.dtype), _dev(p.values, p.dtype), _dev(p.surprisal),
                                    _dev(p.n_tokens), _dev(p.omega[:, :c["sketch"]].copy()), ws)
    torch.cuda.synchronize()
    assert ws.status() == 0, f"builder error bits {ws.status():#x}"
    host = {}
    for k, v in cache.items():
        if v.dtype == torch.bfloat16:
            host[k] = v.view(torch.int16).cpu().numpy().view(np.uint16)
        else:
            host[k] = v.cpu().numpy()
    return host, {k: v.cpu().numpy() for k, v in seg.items() if not k.startswith("_")}, lay


def _orthonormal_err(M):
    return np.abs(M.T @ M - np.eye(M.shape[1])).max() if M.size else 0.0


@pytest.mark.parametrize("name,c", BUILD_CASES, ids=[c[0] for c in BUILD_CASES])
def test_build_matches_oracle(S, name, c):
    banner(f"build {name}")
    dt, d = c["dtype"], c["d"]
    p = make_prefill(len(c["n"]), c["Hkv"], d, c["n"], dtype=dt, spike_every=90, true_rank=20, noise=0.05,
                     sketch=48, seed=74)
    # one span of identical rows (rank one) and one of zeros (rank zero) in sequence 0
    anchors0, spans0 = oracle.segment(p.surprisal[0], int(p.n_tokens[0]), 1.0, c["min_span"], c["window"])
    assert len(spans0) >= 3
    s1, L1 = spans0[1]
    p.keys[0, :, s1:s1 + L1] = p.keys[0, :, s1:s1 + 1]
    s2, L2 = spans0[2]
    p.values[0, :, s2:s2 + L2] = 0
    got, seg, lay = _build(S, p, c)
    _check_segments(seg, p, 1.0, c["min_span"], c["window"], name)
    e = 2 if dt == "bf16" else 4
    gran = 16 // e
    ulp_rel = 2.0 ** -7 if dt == "bf16" else 2.0 ** -23
    rec_rel = 2.0 ** -7 if dt == "bf16" else 1e-5
    orth_tol = 3e-2 if dt == "bf16" else 1e-4
    worst = 0.0
    for b in range(p.surprisal.shape[0]):
        n = int(p.n_tokens[b])
        anchors, spans = oracle.segment(p.surprisal[b], n, 1.0, c["min_span"], c["window"])
        for g in range(c["Hkv"]):
            assert np.array_equal(got["anchor_k"][b, g, :len(anchors)], p.keys[b, g, anchors])
            assert np.array_equal(got["anchor_v"][b, g, :len(anchors)], p.values[b, g, anchors])
        for S_, (s0, L) in enumerate(spans):
            assert got["span_len"][b, S_] == L
            ls = got["span_logsize"][b, S_]
            assert abs(ls - math.log(L)) <= 2 * np.spacing(max(math.log(L), 1e-300)), (b, S_, ls)
            h = p.surprisal[b, s0:s0 + L]
            for g in range(c["Hkv"]):
                for side, src in (("K", p.keys), ("V", p.values)):
                    X = oracle.widen(src[b, g, s0:s0 + L], dt)
                    mx = max(np.abs(X).max(), 1e-30)
                    ref = oracle.weighted_summary(X, h)
                    summ = oracle.widen(got["sum_" + side.lower()][b, g, S_], dt)
                    assert np.all(np.abs(summ - ref) <= ulp_rel * np.abs(ref) + 1e-4 * mx), (name, b, g, S_, side)
                    w = int(lay["block_rank"][b, g, S_])
                    rk, rv = w & 0xFFFF, w >> 16
                    r = min(L, d, c["rank"])
                    assert rk == rv == -(-r // gran) * gran
                    blk = oracle.read_span_block(got["factors"], int(lay["block_off"][b, g, S_]), L, rk, d, dt, rv)
                    U, sg, Vt = blk["U" + side], blk["s" + side], blk["Vt" + side]
                    assert np.all(sg[r:] == 0) and np.all(U[:, r:] == 0) and np.all(Vt[r:] == 0)
                    assert np.all(sg >= 0)
                    full = np.linalg.svd(X, compute_uv=False)
                    opt = math.sqrt(np.sum(full[r:] ** 2))
                    err = np.linalg.norm(X - oracle.reconstruct(U, sg, Vt))
                    nx = np.linalg.norm(X)
                    assert err <= c.get("bound", 1.25) * opt + rec_rel * nx + 1e-30, (name, b, g, S_, side, err,
                                                                                     opt, nx)
                    worst = max(worst, (err - opt) / max(nx, 1e-30))
                    live = sg > 1e-3 * max(sg.max(initial=0), 1e-30)
                    if live.any():
                        assert _orthonormal_err(U[:, live]) <= orth_tol, (name, b, g, S_, side)
                        assert _orthonormal_err(Vt[live].T) <= orth_tol, (name, b, g, S_, side)
    banner(f"build {name}: worst excess reconstruction error {worst:.2e} of ||X||")


@pytest.mark.parametrize("power", [0, 1])
def test_build_is_deterministic(S, power):
    """The builder sums in fixed orders only (no atomics in the arithmetic): two builds of
    the same layer give the same bytes in every output, factors included."""
    banner(f"build determinism, power {power}")
    c = dict(dtype="bf16", d=128, Hkv=2, n=[2600, 1900], rank=32, sketch=40, min_span=4, window=64,
             power=power)
    p = make_prefill(2, 2, 128, c["n"], dtype="bf16", spike_every=120, true_rank=24, noise=0.05,
                     sketch=40, seed=78)
    first, seg1, lay1 = _build(S, p, c)
    second, seg2, lay2 = _build(S, p, c)
    assert lay1["factors_bytes"] == lay2["factors_bytes"]
    for key in seg1:
        assert np.array_equal(seg1[key], seg2[key]), key
    for key in first:
        assert np.array_equal(first[key], second[key]), f"{key} differs between two builds"


def test_build_rejects_tables_past_n_tokens(S):
    """Anchor indices and spans past a sequence's own token count are skipped and flagged
    (error bit 4); everything inside is built as usual."""
    import torch
    banner("build: tables past n_tokens")
    c = dict(dtype="f32", d=64, Hkv=1, n=[900, 600], rank=8, sketch=12, min_span=4, window=16)
    p = make_prefill(2, 1, 64, c["n"], dtype="f32", spike_every=60, seed=77)
    bd = _bdims(S, p, 1, 64, rank=8, sketch=12, min_span=4, window=16)
    dims = S.make_dims(batch=1, n_q_heads=1, n_kv_heads=1, head_dim=64, rank=8, top_k=1, max_anchors=1,
                       max_spans=1, max_span_len=1, dtype="f32", softmax_scale=1.0)
    ws = S.Workspace(dims)
    keys, values, surp = _dev(p.keys), _dev(p.values), _dev(p.surprisal)
    seg = S.segment(bd, surp, _dev(p.n_tokens))
    torch.cuda.synchronize()
    ns, na = seg["n_spans"].cpu().numpy(), seg["n_anchors"].cpu().numpy()
    span_len = seg["span_len"].cpu().numpy()
    off, _, nbytes = S.build_layout(bd, int(ns.max()), ns, span_len)
    # sequence 0 claims 50 tokens fewer than were segmented: its tail anchors fall outside
    short = p.n_tokens.copy()
    short[0] -= 50
    cache = S.build_cache(bd, keys, values, surp, _dev(short), seg, _dev(p.omega[:, :12].copy()), int(na.max()),
                          int(ns.max()), torch.from_numpy(off).cuda(), nbytes, ws)
    torch.cuda.synchronize()
    assert ws.status() == 4
    assert ws.status() == 0                                   # read and cleared
    anchors, _ = oracle.segment(p.surprisal[1], int(p.n_tokens[1]), 1.0, 4, 16)
    got = cache["anchor_k"].cpu().numpy()
    assert np.array_equal(got[1, 0, :len(anchors)], p.keys[1, 0, anchors])
    anchors0, _ = oracle.segment(p.surprisal[0], int(p.n_tokens[0]), 1.0, 4, 16)
    inside = [i for i, t in enumerate(anchors0) if t < short[0]]
    assert np.array_equal(got[0, 0, inside], p.keys[0, 0, [anchors0[i] for i in inside]])


def test_build_layout_and_validate(S):
    """The built cache passes the library's own cache validation with its block ranks."""
    banner("build layout + validate")
    c = dict(dtype="bf16", d=64, Hkv=2, n=[1000, 700], rank=16, sketch=24, min_span=4, window=32)
    p = make_prefill(2, 2, 64, c["n"], dtype="bf16", spike_every=80, seed=75)
    got, seg, lay = _build(S, p, c)
    q = rng(76).standard_normal((2, 4, 64)).astype(np.float32)
    arrays = dict(q=oracle.narrow(q, "bf16"), anchor_k=got["anchor_k"], anchor_v=got["anchor_v"],
                  n_anchors=got["n_anchors"], sum_k=got["sum_k"], sum_v=got["sum_v"], n_spans=got["n_spans"],
                  span_len=got["span_len"], span_logsize=got["span_logsize"], factors=got["factors"],
                  block_off=got["block_off"], block_rank=got["block_rank"])
    dims = S.make_dims(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=16, top_k=4,
                       max_anchors=lay["max_anchors"], max_spans=lay["max_spans"],
                       max_span_len=lay["max_span_len"], dtype="bf16", softmax_scale=0.125)
    S.validate_cache(dims, arrays)


E2E_CASES = [
    ("f32-d128", dict(dtype="f32", d=128, Hkv=2, Hq=8, n=[2500, 1700], rank=32, sketch=40, min_span=8,
                      window=128, top_k=5)),
    ("bf16-d128", dict(dtype="bf16", d=128, Hkv=2, Hq=8, n=[2500, 1700], rank=32, sketch=40, min_span=8,
                       window=128, top_k=5)),
    ("bf16-d64-g4", dict(dtype="bf16", d=64, Hkv=1, Hq=4, n=[3000], rank=16, sketch=24, min_span=4,
                         window=64, top_k=3)),
]


@pytest.mark.parametrize("name,c", E2E_CASES, ids=[c[0] for c in E2E_CASES])
def test_decode_on_built_cache(S, name, c):
    import torch
    banner(f"decode on built cache {name}")
    dt, d = c["dtype"], c["d"]
    true_rank = min(12, c["rank"])
    p = make_prefill(len(c["n"]), c["Hkv"], d, c["n"], dtype=dt, spike_every=120, true_rank=true_rank,
                     noise=0.0, sketch=48, seed=77)
    got, seg, lay = _build(S, p, c)
    ref_cache = oracle.build_layer_cache(p.keys, p.values, p.surprisal, p.n_tokens, alpha=1.0,
                                         min_span=c["min_span"], window=c["window"], r_max=c["rank"], dtype=dt)
    B = len(c["n"])
    scale = 1.0 / math.sqrt(d)
    q = oracle.narrow(rng(78).standard_normal((B, c["Hq"], d)), dt)
    res = oracle.decode_step(q, ref_cache["anchor_k"], ref_cache["anchor_v"], ref_cache["n_anchors"],
                             ref_cache["sum_k"], ref_cache["sum_v"], ref_cache["n_spans"], ref_cache["span_len"],
                             ref_cache["span_logsize"], ref_cache["factors"], ref_cache["block_off"],
                             rank=c["rank"], top_k=c["top_k"], softmax_scale=scale, dtype=dt,
                             block_rank=ref_cache["block_rank"])
    dev = {}
    for k in ("anchor_k", "anchor_v", "sum_k", "sum_v"):
        dev[k] = _dev(got[k], dt)
    for k in ("n_anchors", "n_spans", "span_len", "span_logsize", "factors", "block_off", "block_rank"):
        dev[k] = _dev(got[k])
    dev["q"] = _dev(q, dt)
    cache = S.DeviceCache(dev, dt)
    dims = S.make_dims(batch=B, n_q_heads=c["Hq"], n_kv_heads=c["Hkv"], head_dim=d, rank=c["rank"],
                       top_k=c["top_k"], max_anchors=lay["max_anchors"], max_spans=lay["max_spans"],
                       max_span_len=lay["max_span_len"], dtype=dt, softmax_scale=scale)
    ws = S.Workspace(dims)
    sel, out = S.decode_step(dims, cache, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    sel = sel.cpu().numpy()
    keys, k = res["keys"], c["top_k"]
    G = c["Hq"] // c["Hkv"]
    got_out, ref_out = out_to_f64(out), res["out"]
    checked = 0
    for b in range(B):
        m = int(ref_cache["n_spans"][b])
        for g in range(c["Hkv"]):
            srt = np.sort(keys[b, g, :m])[::-1]
            if m > k and abs(srt[k - 1] - srt[k]) < 1e-2:
                continue            # a near tie: summaries may round apart by one ulp
            kk = min(k, m)
            assert sorted(sel[b, g, :kk].tolist()) == sorted(res["sel"][b, g, :kk].tolist()), (name, b, g)
            assert_out_close(got_out[b, g * G:(g + 1) * G], ref_out[b, g * G:(g + 1) * G], dt, f"{name} b{b} g{g}")
            checked += 1
    assert checked > 0


def test_build_full_size_128k_x4_sampled(S):
    """The builder in the launch configuration of the prefill bench (B 4, Hkv 8, d 128, 131072
    tokens, bf16, R_max 32, sketch 40, one subspace iteration; head g holds the sequence's
    generated stream with its feature columns rotated by 8 g): segmentation bit for bit,
    anchors and span tables, and 24 sampled span sides against the optimal truncated SVD."""
    import torch
    banner("build 131072 x 4 x 8 heads, sampled spans")
    B, Hkv, d, N, R, l = 4, 8, 128, 131072, 32, 40
    p = make_prefill(B, 1, d, N, dtype="bf16", spike_every=170, true_rank=24, noise=0.02, sketch=l, seed=5)
    keys1, vals1 = p.keys, p.values                                  # [B][1][N][d]
    rot = lambda a: np.concatenate([np.roll(a, 8 * g, axis=3) for g in range(Hkv)], axis=1)
    keys, values = rot(keys1), rot(vals1)
    bd = S.make_build_dims(batch=B, n_kv_heads=Hkv, head_dim=d, max_tokens=N, rank=R, sketch=l, min_span=16,
                           window=512, dtype="bf16", power=1)
    wd = S.make_dims(batch=1, n_q_heads=1, n_kv_heads=1, head_dim=64, rank=8, top_k=1, max_anchors=1,
                     max_spans=1, max_span_len=1, dtype="f32", softmax_scale=1.0)
    ws = S.Workspace(wd)
    cache, seg, lay = S.build_layer(bd, _dev(keys, "bf16"), _dev(values, "bf16"), _dev(p.surprisal),
                                    _dev(p.n_tokens), _dev(p.omega), ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    segh = {k: v.cpu().numpy() for k, v in seg.items() if not k.startswith("_")}
    _check_segments(segh, p, 1.0, 16, 512, "full size")
    factors = cache["factors"].cpu().numpy()
    span_len = cache["span_len"].cpu().numpy()
    ak = cache["anchor_k"].view(torch.int16).cpu().numpy().view(np.uint16)
    g_ = np.random.default_rng(99)
    worst = 0.0
    for _ in range(24):
        b = int(g_.integers(B))
        anchors, spans = oracle.segment(p.surprisal[b], N, 1.0, 16, 512)
        g = int(g_.integers(Hkv))
        assert np.array_equal(ak[b, g, :len(anchors)], keys[b, g, anchors])
        S_ = int(g_.integers(len(spans)))
        s0, L = spans[S_]
        assert span_len[b, S_] == L
        side, src = (("K", keys), ("V", values))[int(g_.integers(2))]
        w = int(lay["block_rank"][b, g, S_])
        rk, rv = w & 0xFFFF, w >> 16
        blk = oracle.read_span_block(factors, int(lay["block_off"][b, g, S_]), L, rk, d, "bf16", rv)
        X = oracle.widen(src[b, g, s0:s0 + L], "bf16")
        r = min(L, d, R)
        full = np.linalg.svd(X, compute_uv=False)
        opt = math.sqrt(np.sum(full[r:] ** 2))
        err = np.linalg.norm(X - oracle.reconstruct(blk["U" + side], blk["s" + side], blk["Vt" + side]))
        nx = np.linalg.norm(X)
        assert err <= 1.25 * opt + 2.0 ** -7 * nx, (b, g, S_, side, err, opt, nx)
        worst = max(worst, (err - opt) / nx)
    banner(f"full size: worst excess reconstruction error {worst:.2e} of ||X||")
