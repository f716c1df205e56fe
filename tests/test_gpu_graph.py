"""GPU: several layers captured into one HIP graph (sekv_graph_*), checked against the
eager per-layer calls (bitwise) and against the CPU oracle on every layer.

Each layer has its own independently seeded cache, as in a multi-layer decode step.
Replays are interleaved with eager work and synchronisations, and every replay is
compared with the eager result."""

import numpy as np
import pytest

from synth import WORKLOADS, custom_spec, make_case
from tests.gpu_common import (assert_out_close, banner, case_arrays, dims_for, oracle_result,
                              out_to_f64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


def _layers(spec, n_layers, variant="L"):
    return [make_case(spec, layer=l, variant=variant) for l in range(n_layers)]


def _run_graph_case(S, cases, replays=3):
    import torch
    dev = torch.device("cuda:0")
    dims = dims_for(S, cases[0])
    for c in cases[1:]:
        assert (c.max_spans, c.max_anchors) == (cases[0].max_spans, cases[0].max_anchors)
    dcs = [S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev) for c in cases]
    ws = S.Workspace(dims, dev)
    # eager reference, one call per layer
    eager = [S.decode_step(dims, dc, ws) for dc in dcs]
    torch.cuda.synchronize()
    assert ws.status() == 0
    for l, (c, (sel, out)) in enumerate(zip(cases, eager)):
        ref = oracle_result(c)
        assert np.array_equal(sel.cpu().numpy(), ref["sel"]), f"layer {l}: selection differs"
        assert_out_close(out_to_f64(out), ref["out"], c.dtype, where=f"layer {l}")
    g = S.LayerGraph(dims, dcs, ws)
    try:
        for rep in range(replays):
            g.sel.fill_(-7)
            g.out.zero_()
            torch.cuda.synchronize()
            g.launch()
            torch.cuda.synchronize()
            assert ws.status() == 0
            for l, (sel, out) in enumerate(eager):
                assert torch.equal(g.sel[l], sel), f"replay {rep} layer {l}: selection differs"
                assert torch.equal(g.out[l].view(torch.uint8) if out.dtype == torch.bfloat16
                                   else g.out[l], out.view(torch.uint8)
                                   if out.dtype == torch.bfloat16 else out), \
                    f"replay {rep} layer {l}: output differs from the eager call"
            # eager work on the same workspace between replays
            S.decode_step(dims, dcs[rep % len(dcs)], ws)
            torch.cuda.synchronize()
    finally:
        g.destroy()


def test_graph_small_layers(S):
    banner("graph: 4 small bf16 layers")
    spec = custom_spec(batch=4, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16, top_k=4,
                       context=3000, n_prefix_anchors=64, window=128, dtype="bf16", seed=41,
                       span_min=32, span_max=256, n_layers=4)
    _run_graph_case(S, _layers(spec, 4))


def test_graph_small_layers_f32_planted(S):
    banner("graph: 3 small f32 layers, planted")
    spec = custom_spec(batch=2, n_q_heads=8, n_kv_heads=4, head_dim=64, rank=8, top_k=3,
                       context=2000, n_prefix_anchors=32, window=0, dtype="f32", seed=42,
                       span_min=16, span_max=96, n_layers=3)
    _run_graph_case(S, _layers(spec, 3, variant="N"), replays=2)


def test_graph_32layer_b32_shapes_two_layers(S):
    """Two independently seeded layers at the 32-layer workload's per-layer shape
    (batch 32, 32K context, rank 16, top-8)."""
    banner("graph: 32-layer batch-32 shapes, 2 layers: generating")
    cases = _layers(WORKLOADS["llama3-8b-32layer-32k-b32"], 2)
    banner("graph: 32-layer batch-32 shapes: running")
    _run_graph_case(S, cases, replays=2)


def test_graph_32layer_b32_planted_two_layers(S):
    """The planted-needle variant at the 32-layer workload's per-layer shape, 2 layers."""
    banner("graph: 32-layer batch-32 shapes, planted, 2 layers: generating")
    cases = _layers(WORKLOADS["llama3-8b-32layer-32k-b32"], 2, variant="N")
    banner("graph: 32-layer batch-32 shapes, planted: running")
    _run_graph_case(S, cases, replays=2)


@pytest.mark.slow
def test_graph_32layer_b32_all_32_seeded_layers(S):
    """The whole 32-layer step (batch 32, 32K context, rank 16, top-8): 32 independently
    seeded layers replayed through one 32-node graph; every layer's selection bit for bit
    and its output against the oracle, and every replay against the first."""
    import torch
    spec = WORKLOADS["llama3-8b-32layer-32k-b32"]
    dev = torch.device("cuda:0")
    dcs, refs, dims = [], [], None
    for l in range(spec.n_layers):
        c = make_case(spec, layer=l)
        if dims is None:
            dims = dims_for(S, c)
        else:
            assert (c.max_spans, c.max_anchors) == (dims.max_spans, dims.max_anchors)
            dims.max_span_len = max(dims.max_span_len, c.max_span_len)
        dcs.append(S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev))
        ref = oracle_result(c)
        refs.append((ref["sel"], ref["out"]))
        del c
        banner(f"graph: 32 seeded layers: layer {l} generated and checked by the oracle")
    ws = S.Workspace(dims, dev)
    g = S.LayerGraph(dims, dcs, ws)
    try:
        first = None
        for rep in range(2):
            sel, out = g.launch()
            torch.cuda.synchronize()
            assert ws.status() == 0
            if first is None:
                first = (sel.clone(), out.clone())
                for l, (rs, ro) in enumerate(refs):
                    assert np.array_equal(sel[l].cpu().numpy(), rs), f"layer {l}: selection differs"
                    assert_out_close(out_to_f64(out[l]), ro, "bf16", where=f"layer {l}")
            else:
                assert torch.equal(sel, first[0]) and torch.equal(out.view(torch.uint8),
                                                                  first[1].view(torch.uint8))
            banner(f"graph: 32 seeded layers: replay {rep} checked")
    finally:
        g.destroy()


def test_graph_rejects_bad_layers(S):
    import torch
    dev = torch.device("cuda:0")
    spec = custom_spec(batch=1, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8, top_k=2,
                       context=600, dtype="f32", seed=43)
    c = make_case(spec)
    dims = dims_for(S, c)
    dc = S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev)
    ws = S.Workspace(dims, dev)
    bad = S.DeviceCache(dict(dc.t), c.dtype)
    bad.t["sum_k"] = torch.empty(0, device=dev)         # NULL pointer for one layer
    with pytest.raises(S.SekvError) as ei:
        S.LayerGraph(dims, [dc, bad], ws)
    assert ei.value.status == S.SEKV_ERR_INVALID_ARG and "layer 1" in str(ei.value)
