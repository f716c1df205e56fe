"""GPU parity of the learned selection rule (sekv_route_gated, sekv_decode_step_gated).

Against the oracle on the same seeded inputs: the pre-sigmoid gates bit for bit
(float64), the selection bit for bit, and the step's output within max-abs 2e-2
(bf16 output) or 1e-4 (float32 output) plus relative and cosine checks.
"""

import numpy as np
import pytest

import oracle
from synth import NO_BUDGET, WORKLOADS, custom_spec, make_case, make_gate
from tests.gpu_common import assert_out_close, banner, case_arrays, dims_for, out_to_f64
from tests.helpers import oracle_kwargs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


def _oracle(case, gate, k, budget):
    kw = oracle_kwargs(case)
    kw.pop("top_k")
    return oracle.decode_step_gated(**kw, proj=gate.proj, sum_route=gate.sum_route,
                                    thresholds=gate.thresholds, max_zoom=k, budget_tokens=budget)


def _oracle_selection(case, gate, k, budget):
    """Gates and selection only (no attention): for the large-span-count cases."""
    s = case.spec
    qd = oracle.widen(case.q, s.dtype)
    qp = oracle.project_queries(qd, oracle.widen(gate.proj, s.dtype))
    x = oracle.gate_logits(qp, oracle.widen(gate.sum_route, s.dtype), case.span_logsize, case.n_spans)
    sel = oracle.gated_selection(x, gate.thresholds, case.span_len, case.n_spans, s.n_kv_heads, k, budget)
    return x, sel


def _assert_bits(got, ref, what):
    got = np.asarray(got)
    if not np.array_equal(got, ref):
        bad = got != ref
        fin = bad & np.isfinite(ref)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} differ, max |diff| "
                             f"{np.max(np.abs(got[fin] - ref[fin])) if fin.any() else 'n/a'}")


def _upload(S, case, gate, budget, dev):
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dg = S.DeviceGate.from_arrays(gate.route_dim, gate.proj, gate.sum_route, gate.thresholds, budget,
                                  case.dtype, dev)
    return dc, dg


def _ragged(case):
    if case.spec.batch >= 2:
        case.n_spans = case.n_spans.copy()
        case.n_spans[1] = 0
    if case.spec.batch >= 3:
        case.n_spans[2] = max(1, int(case.n_spans[2]) // 4)
    return case


CASES = [
    # name, spec overrides, route_dim, tau, k, budget, out_dtype
    ("f32-g2-d64-dr8", dict(dtype="f32", n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8, context=1500,
                            span_min=8, span_max=48, seed=51), 8, "spread", 4, 60, None),
    ("bf16-g4-d128-dr32-ragged", dict(dtype="bf16", batch=3, n_q_heads=8, n_kv_heads=2, head_dim=128,
                                      rank=16, context=3000, span_min=16, span_max=120, seed=52),
     32, "spread", 8, NO_BUDGET, None),
    ("f32-g8-d128-dr64", dict(dtype="f32", n_q_heads=16, n_kv_heads=2, head_dim=128, rank=8,
                              context=2500, span_min=10, span_max=90, seed=53), 64, "permissive", 6, 250, None),
    ("bf16-g1-d64-dr16-k64", dict(dtype="bf16", n_q_heads=2, n_kv_heads=2, head_dim=64, rank=8,
                                  context=6000, span_min=8, span_max=60, seed=54), 16, "spread", 64, 2000, "f32"),
    ("bf16-g4-multichunk", dict(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=64, rank=8,
                                context=20000, span_min=8, span_max=40, seed=55), 32, "spread", 16, 300, None),
    ("bf16-g2-planted", dict(dtype="bf16", n_q_heads=4, n_kv_heads=2, head_dim=128, rank=16,
                             context=4000, span_min=16, span_max=100, seed=56, variant="N"),
     32, "permissive", 4, NO_BUDGET, None),
]


@pytest.mark.parametrize("name,spec,dr,tau,k,budget,out_dtype", CASES, ids=[c[0] for c in CASES])
def test_gated_step_matches_oracle(S, name, spec, dr, tau, k, budget, out_dtype):
    import torch
    spec = dict(spec)
    variant = spec.pop("variant", "L")
    banner(f"gated {name}: generating")
    case = make_case(custom_spec(top_k=k, **spec), variant=variant)
    if "ragged" in name:
        case = _ragged(case)
    gate = make_gate(case, route_dim=dr, tau=tau, budget_tokens=budget)
    ref = _oracle(case, gate, k, budget)
    dev = torch.device("cuda:0")
    dc, dg = _upload(S, case, gate, budget, dev)
    dims = dims_for(S, case, top_k=k, out_dtype=out_dtype)
    ws = S.Workspace(dims, dev)
    banner(f"gated {name}: route_gated")
    sel, lg = S.route_gated(dims, dc, dg, ws, want_logits=True)
    torch.cuda.synchronize()
    _assert_bits(lg.cpu().numpy(), ref["gate_logits"], "gate logits")
    assert np.array_equal(sel.cpu().numpy(), ref["sel"]), "selection differs"
    banner(f"gated {name}: decode_step_gated")
    sel2, out = S.decode_step_gated(dims, dc, dg, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert torch.equal(sel2, sel)
    od = out_dtype or case.dtype
    assert_out_close(out_to_f64(out), ref["out"], od, where=name)


def test_gated_many_spans_large_chunks(S):
    """10 000 spans with k = 64: chunks of 512 spans, 20 chunks, 1280 candidates per pair."""
    import torch
    banner("gated many spans: generating")
    case = make_case(custom_spec(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=64, rank=8, top_k=64,
                                 context=80000 + 64, n_prefix_anchors=64, span_min=8, span_max=8,
                                 seed=57))
    assert case.max_spans == 10000
    gate = make_gate(case, route_dim=16, tau="spread")
    x, ref_sel = _oracle_selection(case, gate, 64, 300)
    dev = torch.device("cuda:0")
    dc, dg = _upload(S, case, gate, 300, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel, lg = S.route_gated(dims, dc, dg, ws, want_logits=True)
    torch.cuda.synchronize()
    _assert_bits(lg.cpu().numpy(), x, "gate logits")
    assert np.array_equal(sel.cpu().numpy(), ref_sel)
    assert (ref_sel >= 0).sum() > 0


def test_gated_degenerate_rules(S):
    """No budget, no vote, no slots, no sequences."""
    import torch
    case = make_case(custom_spec(dtype="f32", n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8, top_k=5,
                                 context=1500, span_min=8, span_max=40, seed=58))
    gate = make_gate(case, route_dim=8, tau="spread")
    dev = torch.device("cuda:0")
    dc, dg = _upload(S, case, gate, NO_BUDGET, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    # budget 0: nothing expanded; the output is attention over anchors and coarse entries
    ref0 = _oracle(case, gate, 5, 0)
    assert (ref0["sel"] == -1).all()
    sel, out = S.decode_step_gated(dims, dc, S.DeviceGate(8, dg.proj, dg.sum_route, dg.thresholds, 0), ws)
    torch.cuda.synchronize()
    assert (sel.cpu().numpy() == -1).all()
    assert_out_close(out_to_f64(out), ref0["out"], "f32", where="budget 0")
    # thresholds +inf: no vote
    inf = torch.full_like(dg.thresholds, float("inf"))
    sel, _ = S.route_gated(dims, dc, S.DeviceGate(8, dg.proj, dg.sum_route, inf, NO_BUDGET), ws)
    torch.cuda.synchronize()
    assert (sel.cpu().numpy() == -1).all()
    # top_k = 0: no selection slots, the gates are still written
    dims0 = dims_for(S, case, top_k=0)
    ws0 = S.Workspace(dims0, dev)
    x_ref, _ = _oracle_selection(case, gate, 0, NO_BUDGET)
    _, lg = S.route_gated(dims0, dc, dg, ws0, want_logits=True)
    torch.cuda.synchronize()
    _assert_bits(lg.cpu().numpy(), x_ref, "gate logits")
    # invalid gate arguments are refused on the host
    with pytest.raises(S.SekvError):
        S.route_gated(dims, dc, S.DeviceGate(12, dg.proj, dg.sum_route, dg.thresholds, 10), ws)
    with pytest.raises(S.SekvError):
        S.route_gated(dims, dc, S.DeviceGate(8, dg.proj, dg.sum_route, dg.thresholds, -1), ws)


def test_gated_workspace_shared_with_topk_step(S):
    """Gated and top-k steps alternate on one workspace; every call gives its own bits."""
    import torch
    case = make_case(custom_spec(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16, top_k=6,
                                 context=6000, span_min=16, span_max=90, seed=59))
    gate = make_gate(case, route_dim=32, tau="spread", budget_tokens=400)
    dev = torch.device("cuda:0")
    dc, dg = _upload(S, case, gate, 400, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    ref_g = _oracle(case, gate, 6, 400)
    ref_t = oracle.decode_step(**oracle_kwargs(case))
    first = None
    for it in range(3):
        gsel, gout = S.decode_step_gated(dims, dc, dg, ws)
        tsel, tout = S.decode_step(dims, dc, ws)
        torch.cuda.synchronize()
        assert ws.status() == 0
        assert np.array_equal(gsel.cpu().numpy(), ref_g["sel"]), f"gated selection, call {it}"
        assert np.array_equal(tsel.cpu().numpy(), ref_t["sel"]), f"top-k selection, call {it}"
        if first is None:
            first = (gout.clone(), tout.clone())
            assert_out_close(out_to_f64(gout), ref_g["out"], "bf16", where="gated")
            assert_out_close(out_to_f64(tout), ref_t["out"], "bf16", where="top-k")
        else:
            assert torch.equal(gout, first[0]) and torch.equal(tout, first[1])


def test_gated_step_in_a_graph(S):
    """The gated step (selection kernel, then the step in attend mode) captured into a HIP
    graph: several replays over two cache copies, with eager calls on the same workspace in
    between, each bit for bit equal to the eager call, whose selection is the oracle's."""
    import torch
    case = make_case(custom_spec(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16, top_k=6,
                                 context=6000, span_min=16, span_max=90, seed=61))
    gate = make_gate(case, route_dim=32, tau="spread", budget_tokens=400)
    dev = torch.device("cuda:0")
    dc, dg = _upload(S, case, gate, 400, dev)
    dc2 = S.DeviceCache({k: v.clone() for k, v in dc.t.items()}, case.dtype)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    ref = _oracle(case, gate, 6, 400)
    stream = torch.cuda.current_stream()
    sel_e, out_e = S.decode_step_gated(dims, dc, dg, ws, stream=stream)   # eager first
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel_e.cpu().numpy(), ref["sel"])
    assert_out_close(out_to_f64(out_e), ref["out"], "bf16", where="gated, eager")
    sels = [torch.empty_like(sel_e) for _ in range(2)]
    outs = [torch.empty_like(out_e) for _ in range(2)]
    cap = torch.cuda.Stream()
    cap.wait_stream(stream)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap):
        for j, c in enumerate((dc, dc2)):
            S.decode_step_gated(dims, c, dg, ws, sel=sels[j], out=outs[j], stream=cap)
    stream.wait_stream(cap)
    for rep in range(4):
        for j in range(2):
            sels[j].fill_(-7)
            outs[j].zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert ws.status() == 0, f"replay {rep}"
        for j in range(2):
            assert torch.equal(sels[j], sel_e), f"replay {rep}, copy {j}: selection"
            assert torch.equal(outs[j], out_e), f"replay {rep}, copy {j}: output"
        e_sel, e_out = S.decode_step_gated(dims, dc2, dg, ws, stream=stream)
        t_sel, t_out = S.decode_step(dims, dc, ws, stream=stream)
        torch.cuda.synchronize()
        assert torch.equal(e_out, out_e) and torch.equal(e_sel, sel_e), f"eager call after replay {rep}"
    del graph


@pytest.mark.parametrize("budget", [4096, NO_BUDGET])
def test_gated_layer_128k_b4_full_size(S, budget):
    """The 128K-context, batch-4 layer at full size under the learned rule (tau = 0.05 for
    every head, the paper's initialisation): every gate, selection and output row."""
    import torch
    banner(f"gated 128K x 4, budget {budget}: generating")
    case = make_case(WORKLOADS["llama3-8b-layer-128k-b4"], variant="N")
    gate = make_gate(case, route_dim=32, tau="permissive", budget_tokens=budget)
    banner("gated 128K x 4: oracle")
    ref = _oracle(case, gate, case.spec.top_k, budget)
    dev = torch.device("cuda:0")
    dc, dg = _upload(S, case, gate, budget, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    banner("gated 128K x 4: route_gated + decode_step_gated")
    sel, lg = S.route_gated(dims, dc, dg, ws, want_logits=True)
    sel2, out = S.decode_step_gated(dims, dc, dg, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    _assert_bits(lg.cpu().numpy(), ref["gate_logits"], "gate logits")
    assert np.array_equal(sel.cpu().numpy(), ref["sel"])
    assert torch.equal(sel2, sel)
    assert_out_close(out_to_f64(out), ref["out"], "bf16", where=f"gated 128K x 4 budget {budget}")
