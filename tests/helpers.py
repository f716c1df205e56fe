"""Glue between the synthetic cases and the oracle (test-side only)."""

import numpy as np


def oracle_kwargs(case, top_k=None):
    s = case.spec
    return dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v,
                n_anchors=case.n_anchors, sum_k=case.sum_k, sum_v=case.sum_v,
                n_spans=case.n_spans, span_len=case.span_len,
                span_logsize=case.span_logsize, factors=case.factors,
                block_off=case.block_off, rank=s.rank,
                top_k=s.top_k if top_k is None else top_k,
                softmax_scale=s.softmax_scale, dtype=s.dtype,
                block_rank=getattr(case, "block_rank", None))


def rng(seed):
    return np.random.default_rng(seed)
