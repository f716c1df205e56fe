"""Host side of the prefill-side builder, on the CPU: dimension checks, argument checks that
fail before any device call, and the factor-arena layout (sekv_build_layout, host only)
against a layout computed here from the rule: rank min(|S|, d, R_max) rounded up to the
16-byte granule, block bytes 2 (|S| + 1 + d) r e rounded up to 256, blocks in (b, g, S)
order."""

import os

import numpy as np
import pytest

import oracle
from synth import make_prefill

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2606_31145_amd", "libsekv.so")


@pytest.fixture(scope="module")
def S():
    if not os.path.exists(LIB):
        from paper_2606_31145_amd.build import build
        build()
    from paper_2606_31145_amd import sekv
    return sekv


def _bd(S, **kw):
    base = dict(batch=2, n_kv_heads=2, head_dim=64, max_tokens=1000, rank=32, sketch=40, min_span=8,
                window=16, dtype="bf16", alpha=1.0, sweeps=8, power=1)
    base.update(kw)
    return S.make_build_dims(**base)


def test_workspace_size(S):
    assert S.LIB.sekv_segment_workspace_size(_bd(S)) == 2 * 2000 + 2 * 1002 * 4


@pytest.mark.parametrize("kw", [
    dict(head_dim=96), dict(rank=12), dict(rank=48), dict(rank=0), dict(sketch=30), dict(sketch=41),
    dict(sketch=42), dict(min_span=1), dict(window=-1), dict(sweeps=0), dict(sweeps=33), dict(power=5),
    dict(power=-1), dict(batch=-1), dict(n_kv_heads=0), dict(max_tokens=0), dict(alpha=float("nan")),
    dict(dtype="f32", rank=6),
])
def test_bad_dims_rejected(S, kw):
    assert S.LIB.sekv_segment_workspace_size(_bd(S, **kw)) == 0
    assert S.LIB.sekv_last_error().decode()


def test_f32_granule_accepts_rank_4(S):
    assert S.LIB.sekv_segment_workspace_size(_bd(S, dtype="f32", rank=4, sketch=4)) > 0


def test_null_arguments_rejected_before_launch(S):
    bd = _bd(S)
    with pytest.raises(S.SekvError):
        S._check(S.LIB.sekv_segment(bd, None, None, None, None, None, None, None, None, 0, None))
    with pytest.raises(S.SekvError):
        S._check(S.LIB.sekv_build_cache(bd, *([None] * 10), 4, 4, *([None] * 7), 256, None, None, 0, None))


def _layout_rule(n_spans, span_len, Hkv, d, R, e, M):
    gran = 16 // e
    B = len(n_spans)
    off = np.zeros((B, Hkv, M), np.int64)
    rank = np.zeros((B, Hkv, M), np.int32)
    pos = 0
    for b in range(B):
        for g in range(Hkv):
            for S in range(n_spans[b]):
                L = int(span_len[b][S])
                r = min(L, d, R)
                rs = -(-r // gran) * gran
                off[b, g, S] = pos
                rank[b, g, S] = rs | (rs << 16)
                pos += -(-(2 * (L + 1 + d) * rs * e) // 256) * 256
    return off, rank, max(pos, 256)


@pytest.mark.parametrize("dtype,d,R", [("bf16", 128, 32), ("f32", 64, 8), ("bf16", 64, 40)])
def test_layout_matches_rule(S, dtype, d, R):
    p = make_prefill(3, 1, 16, [1200, 3, 700], dtype="f32", spike_every=50, seed=81)
    N = p.surprisal.shape[1]
    segs = [oracle.segment(p.surprisal[b], int(p.n_tokens[b]), 1.0, 2, 10) for b in range(3)]
    ns = np.array([len(s) for _, s in segs], np.int32)
    sl = np.zeros((3, N), np.int32)
    for b, (_, spans) in enumerate(segs):
        sl[b, :len(spans)] = [L for _, L in spans]
    M = int(ns.max())
    bd = _bd(S, batch=3, n_kv_heads=3, head_dim=d, max_tokens=N, rank=R, sketch=40, dtype=dtype)
    off, rank, nbytes = S.build_layout(bd, M, ns, sl)
    e = 2 if dtype == "bf16" else 4
    ro, rr, rn = _layout_rule(ns, sl, 3, d, R, e, M)
    assert nbytes == rn and np.array_equal(off, ro) and np.array_equal(rank, rr)
    # the built layout satisfies the decode path's host validation of ranks and offsets
    q = np.zeros((3, 3, d), np.float32 if dtype == "f32" else np.uint16)
    st = np.float32 if dtype == "f32" else np.uint16
    arrays = dict(q=q, anchor_k=np.zeros((3, 3, 1, d), st), anchor_v=np.zeros((3, 3, 1, d), st),
                  n_anchors=np.ones(3, np.int32), sum_k=np.zeros((3, 3, M, d), st),
                  sum_v=np.zeros((3, 3, M, d), st), n_spans=ns, span_len=np.maximum(sl[:, :M], 1),
                  span_logsize=np.log(np.maximum(sl[:, :M], 1)).astype(np.float64),
                  factors=np.zeros(nbytes, np.uint8), block_off=off, block_rank=rank)
    rdec = min(x for x in (8, 16, 32, 64) if x >= R)      # the decode step's rank: an upper bound
    dims = S.make_dims(batch=3, n_q_heads=3, n_kv_heads=3, head_dim=d, rank=rdec, top_k=2, max_anchors=1,
                       max_spans=M, max_span_len=int(sl.max()), dtype=dtype, softmax_scale=0.1)
    S.validate_cache(dims, arrays)


def test_layout_rejects_bad_tables(S):
    bd = _bd(S, batch=1, max_tokens=10)
    with pytest.raises(S.SekvError):
        S.build_layout(bd, 2, np.array([3], np.int32), np.full((1, 10), 4, np.int32))   # n_spans > max
    with pytest.raises(S.SekvError):
        S.build_layout(bd, 2, np.array([1], np.int32), np.zeros((1, 10), np.int32))     # empty span
