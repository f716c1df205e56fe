"""Pins of the oracle's per-span adaptive rank (Sec. 3.2 eqs. rank_gates and
key_reconstruction, the deployment-time drop of negligible components, and the
gated approximation error stated with the reconstruction loss in Sec. 3.3).

Checked against the paper's closed form for the gated error, the Eckart-Young
truncation error, and the equivalence of a ragged-rank cache with the same cache
stored at the full rank with the dropped components' sigma set to zero.  Planted
mistakes at the bottom must each break at least one pin.  CPU only.
"""

import numpy as np
import pytest

import oracle
import oracle.sekv_oracle as orc
from synth import case_from_factors, custom_spec, make_case
from synth.cases import from_storage, rank_granule
from tests.helpers import oracle_kwargs, rng


def _exact_svd(M):
    U, s, Vt = np.linalg.svd(M, full_matrices=False)
    return U, s, Vt


def check_gated_error_closed_form():
    """||K - sum_i m_i sigma_i u_i v_i^T||_F^2 = sum_i (1 - m_i)^2 sigma_i^2 for exact factors."""
    g = rng(11)
    for L, d in ((12, 8), (5, 9), (30, 16)):
        K = g.standard_normal((L, d))
        U, s, Vt = _exact_svd(K)
        m = g.uniform(0.0, 1.0, s.size)
        err = np.linalg.norm(K - orc.gated_reconstruct(U, s, Vt, m)) ** 2
        assert abs(err - np.sum((1 - m) ** 2 * s ** 2)) <= 1e-10 * np.sum(s ** 2)


def check_deploy_drop_and_truncation():
    g = rng(12)
    K = g.standard_normal((20, 10))
    U, s, Vt = _exact_svd(K)
    m = g.uniform(0.2, 1.0, s.size)
    keep = m > 0.5
    Ud, sd, Vd = orc.deploy_factors(U, s, Vt, m, keep)
    assert Ud.shape == (20, int(keep.sum())) and sd.shape == (int(keep.sum()),)
    ref = orc.gated_reconstruct(U, s, Vt, np.where(keep, m, 0.0))
    assert np.allclose(orc.reconstruct(Ud, sd, Vd), ref, rtol=0, atol=1e-12)
    # all gates 1, keep the leading r: the best rank-r approximation (Eckart-Young)
    for r in (1, 3, 7):
        Ur, sr, Vr = orc.deploy_factors(U, s, Vt, np.ones(s.size), np.arange(s.size) < r)
        err = np.linalg.norm(K - orc.reconstruct(Ur, sr, Vr)) ** 2
        assert abs(err - np.sum(s[r:] ** 2)) <= 1e-10 * np.sum(s ** 2)


def _adaptive_case(dtype="f32", seed=31, **kw):
    base = dict(dtype=dtype, n_q_heads=4, n_kv_heads=2, head_dim=32, rank=16, top_k=4, context=700,
                span_min=8, span_max=60, seed=seed, rank_mode="adaptive")
    base.update(kw)
    return make_case(custom_spec(**base))


def _parse_block(case, b, g, S):
    """This test's own reading of a ragged block (the layout of the stored cache):
    U_K[|S|][r_K] | sigma_K[r_K] | Vt_K[r_K][d] | U_V[|S|][r_V] | sigma_V[r_V] | Vt_V[r_V][d],
    with r_K | r_V << 16 in the rank table."""
    s = case.spec
    d = s.head_dim
    w = int(case.block_rank[b, g, S])
    ranks = (w & 0xFFFF, w >> 16)
    L = int(case.span_len[b, S])
    et = np.float32 if s.dtype == "f32" else np.uint16
    n = sum(r * (L + 1 + d) for r in ranks)
    raw = np.frombuffer(case.factors.data, dtype=et, count=n, offset=int(case.block_off[b, g, S]))
    x = from_storage(raw, s.dtype)
    out, pos = {}, 0
    for side, r in zip(("K", "V"), ranks):
        out["U" + side] = x[pos:pos + L * r].reshape(L, r); pos += L * r
        out["s" + side] = x[pos:pos + r]; pos += r
        out["Vt" + side] = x[pos:pos + r * d].reshape(r, d); pos += r * d
    return out, ranks


def _padded_equivalent(case):
    """The same cache stored at the full rank, dropped components with sigma = 0."""
    s = case.spec
    R, d = s.rank, s.head_dim
    q = from_storage(case.q, s.dtype)
    B, Hkv = case.block_off.shape[:2]
    ak = [from_storage(case.anchor_k[b, :, :int(case.n_anchors[b])], s.dtype) for b in range(B)]
    av = [from_storage(case.anchor_v[b, :, :int(case.n_anchors[b])], s.dtype) for b in range(B)]
    spans = []
    for b in range(B):
        per_b = []
        for S in range(int(case.n_spans[b])):
            heads = []
            for g in range(Hkv):
                f, (rk, rv) = _parse_block(case, b, g, S)
                L = int(case.span_len[b, S])
                padded = {}
                for side, r in (("K", rk), ("V", rv)):
                    Up = np.zeros((L, R)); Up[:, :r] = f["U" + side]
                    sp = np.zeros(R); sp[:r] = f["s" + side]
                    Vp = np.zeros((R, d)); Vp[:r] = f["Vt" + side]
                    padded.update({"U" + side: Up, "s" + side: sp, "Vt" + side: Vp})
                heads.append(padded)
            per_b.append(heads)
        spans.append(per_b)
    return case_from_factors(q, ak, av, spans, dtype=s.dtype, top_k=s.top_k,
                             sum_k=from_storage(case.sum_k, s.dtype), sum_v=from_storage(case.sum_v, s.dtype))


def check_ragged_equals_zero_padded():
    for dtype in ("f32", "bf16"):
        case = _adaptive_case(dtype=dtype)
        gr = rank_granule(dtype)
        rk = case.block_rank & 0xFFFF
        rv = case.block_rank >> 16
        live = case.block_rank != 0
        assert np.all(rk[live] % gr == 0) and np.all(rv[live] % gr == 0)
        assert np.all((rk[live] >= gr) & (rk[live] <= case.spec.rank))
        assert len(np.unique(rk[live])) > 1 and np.any(rk[live] != rv[live])
        ref = orc.decode_step(**oracle_kwargs(case))
        pad = _padded_equivalent(case)
        got = orc.decode_step(**oracle_kwargs(pad))
        assert np.array_equal(got["sel"], ref["sel"])
        assert np.allclose(got["out"], ref["out"], rtol=1e-12, atol=1e-14)


def check_full_rank_table_is_no_table():
    case = make_case(custom_spec(dtype="f32", n_q_heads=4, n_kv_heads=2, head_dim=32, rank=8, top_k=3,
                                 context=500, span_min=8, span_max=40, seed=33))
    R = case.spec.rank
    kw = oracle_kwargs(case)
    a = orc.decode_step(**kw)
    table = np.where(case.span_len[:, None, :] > 0, R | (R << 16), 0).astype(np.int32)
    table = np.broadcast_to(table, case.block_off.shape).copy()
    b = orc.decode_step(**dict(kw, block_rank=table))
    assert np.array_equal(a["out"], b["out"]) and np.array_equal(a["sel"], b["sel"])


PINS = [check_gated_error_closed_form, check_deploy_drop_and_truncation, check_ragged_equals_zero_padded,
        check_full_rank_table_is_no_table]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_rank_pin(pin):
    pin()


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

_orig_read = orc.read_span_block
_orig_ranks = orc.block_ranks
_orig_gated = orc.gated_reconstruct
_orig_deploy = orc.deploy_factors


def _v_side_uses_k_rank(factors, offset, length, rank, head_dim, dtype, rank_v=None):
    return _orig_read(factors, offset, length, rank, head_dim, dtype, rank_v=rank)


def _swapped_ranks(block_rank, b, g, S, rank):
    rk, rv = _orig_ranks(block_rank, b, g, S, rank)
    return rv, rk


def _gates_squared(U, sigma, Vt, gates):
    return _orig_gated(U, sigma, Vt, np.asarray(gates) ** 2)


def _gate_not_folded(U, sigma, Vt, gates, keep):
    idx = np.flatnonzero(np.asarray(keep, dtype=bool))
    return U[:, idx], sigma[idx], Vt[idx]


MUTANTS = {
    "V side read with the K rank": ("read_span_block", _v_side_uses_k_rank),
    "ranks swapped": ("block_ranks", _swapped_ranks),
    "gates squared": ("gated_reconstruct", _gates_squared),
    "gate not folded into sigma": ("deploy_factors", _gate_not_folded),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_rank_planted_mistake_breaks_a_pin(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(orc, attr, fn)
    monkeypatch.setattr(oracle, attr, fn, raising=False)
    failed = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake: {name}"
