"""Byte accounting against the paper's App. D closed forms (golden fixture) and by hand."""

import json
import os

import numpy as np

from paper_2606_31145_amd import accounting as A

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_appendix_d.json")))


def test_full_kv_bytes_per_token_matches_printed_figure():
    g = GOLD["full_kv_example"]
    per_token = A.mem_fullkv(g["n_layers"], g["n_kv_heads"], g["head_dim"], 1, g["elem_bytes"])
    assert per_token == g["printed_kb_per_token"] * 1024
    total = A.mem_fullkv(g["n_layers"], g["n_kv_heads"], g["head_dim"], g["tokens_128k"], g["elem_bytes"])
    assert total == g["printed_gb_at_128k"] * 2 ** 30


def test_routing_parameter_count_matches_printed_figure():
    g = GOLD["routing_params_example"]
    n = g["n_layers"] * g["n_q_heads"] * g["routing_dim"] * g["head_dim"]
    assert round(n / 1e6, 2) == g["printed_millions"]


def test_span_factor_bytes_and_transfer():
    # r(|S| + d + 1) values per side and per head/layer, keys and values
    assert A.mem_cpu_span(1, 1, 32, 100, 128, 2) == 2 * 32 * (100 + 128 + 1) * 2
    assert A.transfer_bytes(2, 8, 16, [10, 20], 128, 2) == sum(
        2 * 2 * 8 * 16 * (s + 128 + 1) * 2 for s in (10, 20))


def test_step_bytes_by_hand():
    n_anchors = np.array([5, 3])
    n_spans = np.array([4, 2])
    span_len = np.array([[10, 20, 30, 40], [7, 9, 0, 0]])
    sel = np.array([[[2, 0], [1, -1]], [[1, 0], [0, -1]]])          # B=2, Hkv=2, k=2
    r = A.step_bytes(n_q_heads=4, n_kv_heads=2, head_dim=8, rank=4, elem=2, out_elem=4,
                     n_anchors=n_anchors, n_spans=n_spans, span_len=span_len, sel=sel)
    assert r["q"] == 2 * 4 * 8 * 2 and r["out"] == 2 * 4 * 8 * 4
    assert r["anchors"] == 2 * 2 * (5 + 3) * 8 * 2
    assert r["mean_k"] == 2 * (4 + 2) * 8 * 2
    assert r["n_selected"] == 6
    assert r["mean_v"] == (2 * 6 - 6) * 8 * 2
    lens = [30, 10, 20, 9, 7, 7]
    assert r["factors"] == sum(2 * 4 * (L + 8 + 1) * 2 for L in lens)
    assert r["total"] == sum(r[k] for k in ("q", "out", "anchors", "mean_k", "mean_v", "factors", "tables"))


def test_gate_bytes_by_hand():
    g = A.gate_bytes(n_q_heads=4, head_dim=8, route_dim=2, elem=2, n_spans=[3, 1], top_k=2,
                     n_kv_heads=2)
    assert g["q"] == 2 * 4 * 8 * 2
    assert g["proj"] == 4 * 2 * 8 * 2
    assert g["summaries"] == 4 * 4 * 2 * 2
    assert g["tables"] == 4 * 2 + 4 * 12
    assert g["sel"] == 2 * 2 * 2 * 4
    assert g["total"] == sum(g[k] for k in ("q", "proj", "summaries", "tables", "sel"))


def test_step_bytes_with_ranks():
    import numpy as np
    base = dict(n_q_heads=2, n_kv_heads=1, head_dim=4, rank=8, elem=2, out_elem=2,
                n_anchors=[0], n_spans=[2], span_len=np.array([[3, 5]]), sel=np.array([[[1, -1]]]))
    fixed = A.step_bytes(**base)
    assert fixed["factors"] == 2 * 8 * (5 + 4 + 1) * 2
    ragged = A.step_bytes(**base, block_rank=np.array([[[8 | (8 << 16), 4 | (8 << 16)]]]))
    assert ragged["factors"] == (4 + 8) * (5 + 4 + 1) * 2
    assert fixed["total"] - ragged["total"] == fixed["factors"] - ragged["factors"]
