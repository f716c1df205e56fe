"""GPU parity of per-span adaptive ranks: each span block keeps its own r_K, r_V <= rank
(Sec. 3.2, eqs. rank_gates and key_reconstruction, the deployment-time drop).

Every entry point that reads factor blocks -- the fused step, route + attend, the
multi-layer graph, the pinned-host tier in both copy modes and the learned-routing step --
against the CPU oracle on the same seeded ragged-rank caches: selection bit for bit,
outputs within max-abs 2e-2 (bf16 output) or 1e-4 (float32 output) plus relative and
cosine checks; the tier and the graph bitwise against the device-resident stream launch.
"""

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, custom_spec, make_case, make_gate
from synth.cases import block_bytes
from tests.gpu_common import assert_out_close, banner, case_arrays, dims_for, oracle_result, out_to_f64
from tests.helpers import oracle_kwargs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


def _case(**kw):
    variant = kw.pop("variant", "L")
    base = dict(rank_mode="adaptive")
    base.update(kw)
    return make_case(custom_spec(**base), variant=variant)


CASES = [
    ("bf16-d128-r32-g4", dict(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=128, rank=32, top_k=6,
                              context=5000, span_min=16, span_max=200, seed=61)),
    ("f32-d64-r16-g2-N", dict(dtype="f32", n_q_heads=4, n_kv_heads=2, head_dim=64, rank=16, top_k=4,
                              context=3000, span_min=8, span_max=120, seed=62, variant="N")),
    ("bf16-d64-r64-g8", dict(dtype="bf16", n_q_heads=16, n_kv_heads=2, head_dim=64, rank=64, top_k=5,
                             context=4000, span_min=16, span_max=700, seed=63)),
    ("f32-d128-r8-g1", dict(dtype="f32", n_q_heads=2, n_kv_heads=2, head_dim=128, rank=8, top_k=3,
                            context=2000, span_min=8, span_max=80, seed=64)),
    ("bf16-d128-r16-g4-multislot", dict(dtype="bf16", batch=40, n_q_heads=8, n_kv_heads=4, head_dim=128,
                                        rank=16, top_k=7, context=1500, n_prefix_anchors=32, span_min=16,
                                        span_max=120, seed=65)),
]


@pytest.mark.parametrize("name,spec", CASES, ids=[c[0] for c in CASES])
def test_adaptive_rank_step_matches_oracle(S, name, spec):
    import torch
    banner(f"ranks {name}: generating")
    case = _case(**spec)
    assert case.block_rank is not None
    ref = oracle_result(case)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    banner(f"ranks {name}: decode_step")
    sel, out = S.decode_step(dims, dc, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel.cpu().numpy(), ref["sel"])
    assert_out_close(out_to_f64(out), ref["out"], case.dtype, where=name)
    banner(f"ranks {name}: route + attend")
    sel_r, logits = S.route_topk(dims, dc, ws)
    out_r = S.zoom_attend(dims, dc, sel_r, logits, ws)
    out_n = S.zoom_attend(dims, dc, sel_r, None, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert torch.equal(sel_r, sel)
    assert_out_close(out_to_f64(out_r), ref["out"], case.dtype, where=name + " attend")
    assert_out_close(out_to_f64(out_n), ref["out"], case.dtype, where=name + " attend, logits recomputed")


def test_adaptive_rank_graph_and_fixed_table(S):
    """Two ragged-rank layers in one graph, bitwise against eager steps; and a table that
    holds the full rank everywhere gives the bits of no table."""
    import torch
    dev = torch.device("cuda:0")
    spec = custom_spec(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=128, rank=32, top_k=5, context=4000,
                       span_min=16, span_max=200, seed=66, rank_mode="adaptive")
    layers = [make_case(spec, layer=i) for i in range(2)]       # one partition, own values and ranks
    assert not np.array_equal(layers[0].block_rank, layers[1].block_rank)
    dims = dims_for(S, layers[0])
    caches = [S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev) for c in layers]
    ws = S.Workspace(dims, dev)
    eager = [S.decode_step(dims, dc, ws) for dc in caches]
    torch.cuda.synchronize()
    for c, (sel, out) in zip(layers, eager):
        ref = oracle_result(c)
        assert np.array_equal(sel.cpu().numpy(), ref["sel"])
        assert_out_close(out_to_f64(out), ref["out"], "bf16", where="graph layer")
    g = S.LayerGraph(dims, caches, ws)
    try:
        for _ in range(3):
            gsel, gout = g.launch()
            torch.cuda.synchronize()
            assert ws.status() == 0
            for l in range(2):
                assert torch.equal(gsel[l], eager[l][0]) and torch.equal(gout[l], eager[l][1])
    finally:
        g.destroy()
    # full-rank table == no table
    fixed = make_case(custom_spec(dtype="f32", n_q_heads=4, n_kv_heads=2, head_dim=64, rank=16, top_k=4,
                                  context=2500, span_min=8, span_max=100, seed=69))
    R = fixed.spec.rank
    table = np.where(fixed.span_len[:, None, :] > 0, R | (R << 16), 0).astype(np.int32)
    arr = case_arrays(fixed)
    dims_f = dims_for(S, fixed)
    wsf = S.Workspace(dims_f, dev)
    a_sel, a_out = S.decode_step(dims_f, S.DeviceCache.from_arrays(arr, "f32", dev), wsf)
    b_sel, b_out = S.decode_step(dims_f, S.DeviceCache.from_arrays(
        dict(arr, block_rank=np.broadcast_to(table, fixed.block_off.shape).copy()), "f32", dev), wsf)
    torch.cuda.synchronize()
    assert torch.equal(a_sel, b_sel) and torch.equal(a_out, b_out)


@pytest.mark.parametrize("mode", ["gather", "memcpy"])
def test_adaptive_rank_tier(S, mode):
    """The pinned-host tier moves only the kept components: bitwise equal to the device
    path, and the bytes moved are the ragged blocks' bytes."""
    import torch
    banner(f"ranks tier {mode}")
    case = _case(dtype="bf16", batch=3, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=32, top_k=5,
                 context=4000, n_prefix_anchors=64, window=128, span_min=32, span_max=300, seed=70,
                 variant="N")
    dev = torch.device("cuda:0")
    dims = dims_for(S, case)
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    ws = S.Workspace(dims, dev)
    sel_r, logits = S.route_topk(dims, dc, ws)
    out_r = S.zoom_attend(dims, dc, sel_r, logits, ws)
    torch.cuda.synchronize()
    ref = oracle_result(case)
    host = S.HostFactors(case.factors, case.block_off, case.span_len, case.block_rank)
    tier = S.Tier(dims, mode)
    side = torch.cuda.Stream()
    try:
        for step in range(2):
            sel, out = S.decode_step_tiered(dims, dc, host, tier, ws, side=side)
            torch.cuda.synchronize()
            assert ws.status() == 0
            assert np.array_equal(sel.cpu().numpy(), ref["sel"])
            assert torch.equal(out.view(torch.uint8), out_r.view(torch.uint8)), f"step {step}"
            assert_out_close(out_to_f64(out), ref["out"], "bf16", where=f"ranks tier {mode}")
            nbytes, _, _ = tier.last_copy()
            s = ref["sel"]
            raw = tight = 0
            for b in range(s.shape[0]):
                for g in range(s.shape[1]):
                    for x in s[b, g]:
                        if x < 0:
                            continue
                        w = int(case.block_rank[b, g, x])
                        rk, rv = w & 0xFFFF, w >> 16
                        L = int(case.span_len[b, x])
                        raw += block_bytes(L, rk, 128, "bf16", rv)
                        tight += (rk + rv) * (L + 128 + 1) * 2
            assert tight <= nbytes <= raw, (tight, nbytes, raw)
        # a host table without the device table is refused
        with pytest.raises(S.SekvError):
            S.decode_step_tiered(dims, S.DeviceCache({k: v for k, v in dc.t.items() if k != "block_rank"},
                                                     case.dtype), host, tier, ws, side=side)
    finally:
        tier.destroy()


def test_adaptive_rank_invalid_entry_is_skipped_and_flagged(S):
    """A rank-table entry that is not a multiple of the granule: the block is skipped and
    the block-range error bit set; every other pair's output keeps its bits."""
    import torch
    case = _case(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=128, rank=32, top_k=4, context=3000,
                 span_min=16, span_max=150, seed=71)
    ref = oracle_result(case)
    dev = torch.device("cuda:0")
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel0, out0 = S.decode_step(dims, S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev), ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    bad = case.block_rank.copy()
    S0 = int(ref["sel"][0, 1, 0])
    bad[0, 1, S0] = 3 | (8 << 16)                      # r_K = 3: not a multiple of 8
    sel1, out1 = S.decode_step(dims, S.DeviceCache.from_arrays(dict(case_arrays(case), block_rank=bad),
                                                                case.dtype, dev), ws)
    torch.cuda.synchronize()
    assert ws.status() & 2
    assert torch.equal(sel1, sel0)
    assert torch.equal(out1[0, :4], out0[0, :4])        # KV head 0 untouched
    assert not torch.equal(out1[0, 4:], out0[0, 4:])    # KV head 1 lost a zoomed span


def test_adaptive_rank_gated_step(S):
    import torch
    case = _case(dtype="bf16", n_q_heads=8, n_kv_heads=2, head_dim=128, rank=32, top_k=6, context=5000,
                 span_min=16, span_max=200, seed=72)
    gate = make_gate(case, route_dim=32, tau="spread", budget_tokens=600)
    kw = oracle_kwargs(case)
    kw.pop("top_k")
    ref = oracle.decode_step_gated(**kw, proj=gate.proj, sum_route=gate.sum_route, thresholds=gate.thresholds,
                                   max_zoom=6, budget_tokens=600)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dg = S.DeviceGate.from_arrays(32, gate.proj, gate.sum_route, gate.thresholds, 600, case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel, out = S.decode_step_gated(dims, dc, dg, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel.cpu().numpy(), ref["sel"])
    assert_out_close(out_to_f64(out), ref["out"], "bf16", where="gated, adaptive ranks")


def test_adaptive_rank_layer_128k_b4_full_size(S):
    """The 128K x 4 layer with per-span ranks in {8, 16, 24, 32}: every selection and row."""
    import torch
    from dataclasses import replace
    banner("ranks 128K x 4: generating")
    spec = replace(WORKLOADS["llama3-8b-layer-128k-b4"], rank_mode="adaptive")
    case = make_case(spec, variant="N")
    ref = oracle_result(case)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel, out = S.decode_step(dims, dc, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel.cpu().numpy(), ref["sel"])
    assert_out_close(out_to_f64(out), ref["out"], "bf16", where="ranks 128K x 4")
