"""Byte accounting of one SeKV decode step.

Two kinds of figures:

* the paper's closed forms (App. D, "Memory and Complexity Analysis"): full-KV memory
  2 L H_kv d_h n b, per-span CPU storage 2 L H_kv r (|S| + d_h + 1) b, and the per-step
  transfer of the zoomed spans, the same sum over the selected spans;
* the algorithmic HBM bytes of one device-resident decode step: what the method must
  move at least once -- query in, output out, every full-resolution token's key and
  value, every span's coarse mean key (routing), the coarse mean value of every span
  left unexpanded, the factor blocks of the expanded spans, and the span tables.
  Reconstructed tokens are never written, so they cost nothing here.
"""

from __future__ import annotations

import numpy as np


# -- paper closed forms (App. D) ------------------------------------------------------------

def mem_fullkv(n_layers: int, n_kv_heads: int, head_dim: int, n_tokens: int, elem: int) -> int:
    """Full KV cache bytes: 2 L H_kv d_h n b."""
    return 2 * n_layers * n_kv_heads * head_dim * n_tokens * elem


def mem_cpu_span(n_layers: int, n_kv_heads: int, rank: int, span: int, head_dim: int,
                 elem: int) -> int:
    """Low-rank factors of one span for keys and values: 2 L H_kv r (|S| + d_h + 1) b."""
    return 2 * n_layers * n_kv_heads * rank * (span + head_dim + 1) * elem


def transfer_bytes(n_layers: int, n_kv_heads: int, rank: int, spans, head_dim: int,
                   elem: int) -> int:
    """Bytes moved for the zoomed spans of one step: sum over Z_t of mem_cpu_span."""
    return sum(mem_cpu_span(n_layers, n_kv_heads, rank, int(s), head_dim, elem) for s in spans)


# -- one device-resident step ------------------------------------------------------------

def step_bytes(*, n_q_heads: int, n_kv_heads: int, head_dim: int, rank: int, elem: int,
               out_elem: int, n_anchors, n_spans, span_len, sel, block_rank=None) -> dict:
    """Algorithmic HBM bytes of one decode step of one layer, itemised.

    n_anchors [B], n_spans [B], span_len [B][M], sel [B][Hkv][k] (-1 = empty slot);
    block_rank [B][Hkv][M] (r_K | r_V << 16) or None when every block has `rank`.
    """
    n_anchors = np.asarray(n_anchors, dtype=np.int64)
    n_spans = np.asarray(n_spans, dtype=np.int64)
    span_len = np.asarray(span_len, dtype=np.int64)
    sel = np.asarray(sel)
    B = n_anchors.shape[0]
    d, r, Hkv, Hq = head_dim, rank, n_kv_heads, n_q_heads
    q_in = B * Hq * d * elem
    out = B * Hq * d * out_elem
    anchors = int(2 * Hkv * n_anchors.sum() * d * elem)
    mean_k = int(Hkv * n_spans.sum() * d * elem)
    n_sel = int((sel >= 0).sum())
    mean_v = int((Hkv * n_spans.sum() - n_sel) * d * elem)
    factors = 0
    sel_len = []
    for b in range(B):
        for g in range(Hkv):
            for s in sel[b, g]:
                if s >= 0:
                    L = int(span_len[b, s])
                    sel_len.append(L)
                    if block_rank is None:
                        factors += 2 * r * (L + d + 1) * elem
                    else:
                        w = int(block_rank[b, g, s])
                        factors += ((w & 0xFFFF) + (w >> 16)) * (L + d + 1) * elem
    # span tables: n_spans, n_anchors, |S| (int32) and ln|S| (float64) of every span,
    # block offsets (int64) of the expanded spans
    tables = int(8 * B + n_spans.sum() * (4 + 8) + n_sel * 8)
    total = q_in + out + anchors + mean_k + mean_v + factors + tables
    return dict(total=total, q=q_in, out=out, anchors=anchors, mean_k=mean_k, mean_v=mean_v,
                factors=factors, tables=tables, n_selected=n_sel,
                mean_selected_len=float(np.mean(sel_len)) if sel_len else 0.0)


def full_kv_bytes_same_shapes(*, n_kv_heads: int, head_dim: int, elem: int, n_anchors,
                              span_len) -> int:
    """A dense cache of the same tokens (one layer): 2 H_kv d b times every token."""
    tokens = int(np.asarray(n_anchors, dtype=np.int64).sum() +
                 np.asarray(span_len, dtype=np.int64).sum())
    return 2 * n_kv_heads * head_dim * elem * tokens


def gate_bytes(*, n_q_heads: int, head_dim: int, route_dim: int, elem: int, n_spans,
               top_k: int, n_kv_heads: int) -> dict:
    """Algorithmic HBM bytes of the learned-routing selection of one layer, itemised.

    The query in, each query head's projection W (d' x d), the routing summary of every
    live span for every query head (d' values), |S| and ln|S| of every span, and the
    selection out.  The gate values themselves are an optional output and not counted.
    """
    n_spans = np.asarray(n_spans, dtype=np.int64)
    B = n_spans.shape[0]
    q_in = B * n_q_heads * head_dim * elem
    proj = n_q_heads * route_dim * head_dim * elem
    summaries = int(n_q_heads * n_spans.sum() * route_dim * elem)
    tables = int(4 * B + n_spans.sum() * (4 + 8))
    sel = B * n_kv_heads * top_k * 4
    total = q_in + proj + summaries + tables + sel
    return dict(total=total, q=q_in, proj=proj, summaries=summaries, tables=tables, sel=sel)
