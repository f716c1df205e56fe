"""Shared helpers for the GPU tests: upload a synthetic case, run the library, compare."""

import sys

import numpy as np

import oracle
from synth.cases import from_storage
from tests.helpers import oracle_kwargs


def banner(msg):
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def case_arrays(case):
    arr = dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v,
               n_anchors=case.n_anchors, sum_k=case.sum_k, sum_v=case.sum_v,
               n_spans=case.n_spans, span_len=case.span_len, span_logsize=case.span_logsize,
               factors=case.factors, block_off=case.block_off)
    if getattr(case, "block_rank", None) is not None:
        arr["block_rank"] = case.block_rank
    return arr


def dims_for(S, case, out_dtype=None, top_k=None, zoom=0):
    s = case.spec
    return S.make_dims(batch=s.batch, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                       head_dim=s.head_dim, rank=s.rank,
                       top_k=s.top_k if top_k is None else top_k,
                       max_anchors=case.max_anchors, max_spans=case.max_spans,
                       max_span_len=case.max_span_len, dtype=s.dtype,
                       softmax_scale=s.softmax_scale, out_dtype=out_dtype, zoom=zoom)


def oracle_result(case, top_k=None):
    return oracle.decode_step(**oracle_kwargs(case, top_k=top_k))


def out_to_f64(t):
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def assert_out_close(got, ref, out_dtype, where=""):
    """Outputs within the stated tolerances: absolute, relative to the output scale, cosine."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"non-finite output {where}"
    err = np.abs(got - ref)
    scale = max(np.abs(ref).max(), 1e-30)
    if out_dtype == "bf16":
        abs_tol, rel_tol = 2e-2, 2e-2
    else:
        abs_tol, rel_tol = 1e-4, 2e-5
    assert err.max() <= abs_tol, f"max abs err {err.max():.3e} > {abs_tol} {where}"
    assert err.max() / scale <= rel_tol, f"max rel err {err.max() / scale:.3e} > {rel_tol} {where}"
    g2 = got.reshape(-1, got.shape[-1])
    r2 = ref.reshape(-1, ref.shape[-1])
    num = (g2 * r2).sum(-1)
    den = np.linalg.norm(g2, axis=-1) * np.linalg.norm(r2, axis=-1)
    ok = den > 0
    cos = np.ones(len(num))
    cos[ok] = num[ok] / den[ok]
    assert cos.min() >= 0.9999, f"min cosine {cos.min():.6f} {where}"


def min_boundary_gap(res, case):
    """Smallest relative gap between the k-th and (k+1)-th key (informational)."""
    keys = res["keys"]
    k = case.spec.top_k
    gaps = []
    for b in range(keys.shape[0]):
        m = int(case.n_spans[b])
        if m <= k or k == 0:
            continue
        for g in range(keys.shape[1]):
            srt = np.sort(keys[b, g, :m])[::-1]
            gaps.append(abs(srt[k - 1] - srt[k]) / max(abs(srt[k - 1]), 1e-300))
    return min(gaps) if gaps else float("inf")


def ref_logits_f32(res):
    return res["logits"].astype(np.float32)


__all__ = ["banner", "case_arrays", "dims_for", "oracle_result", "out_to_f64", "assert_out_close",
           "min_boundary_gap", "ref_logits_f32", "from_storage"]
