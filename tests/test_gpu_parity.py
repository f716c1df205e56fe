"""GPU parity: every C-ABI entry point against the CPU oracle on the same seeded inputs.

Selection must match bit for bit; outputs within max-abs 2e-2 (bf16 output) or 1e-4
(float32 output), plus relative and cosine checks because the literal caches give
tiny, near-uniform outputs.  Run on an MI355X with the library built in-tree.
"""

import numpy as np
import pytest

from synth import WORKLOADS, custom_spec, make_case
from synth.cases import Case
from tests.gpu_common import (assert_out_close, banner, case_arrays, dims_for, min_boundary_gap,
                              oracle_result, out_to_f64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


def _ragged(case: Case) -> Case:
    """Shrink some sequences: fewer spans, no spans, no anchors, a third of the anchors
    (tables only)."""
    B = case.spec.batch
    if B >= 2:
        case.n_spans = case.n_spans.copy()
        case.n_anchors = case.n_anchors.copy()
        case.n_spans[1] = 0
        if B >= 3:
            case.n_anchors[2] = 0
            case.n_spans[2] = max(1, int(case.n_spans[2]) // 3)
        if B >= 4:
            case.n_spans[3] = min(int(case.n_spans[3]), max(1, case.spec.top_k // 2))
        if B >= 5:
            case.n_anchors[4] = int(case.n_anchors[4]) // 3
    return case


def _custom(name, **kw):
    variant = kw.pop("variant", "L")
    ragged = kw.pop("ragged", False)
    c = make_case(custom_spec(**kw), variant=variant)
    if ragged:
        c = _ragged(c)
    return name, c


def small_cases():
    out = [("tiny-f32-L", make_case(WORKLOADS["tiny-f32"], variant="L")),
           ("tiny-f32-N", make_case(WORKLOADS["tiny-f32"], variant="N")),
           ("layer-32k-L", make_case(WORKLOADS["llama3-8b-layer-32k"], variant="L")),
           ("layer-32k-N", make_case(WORKLOADS["llama3-8b-layer-32k"], variant="N"))]
    out += [
        _custom("g1-bf16-d128-r16", n_q_heads=4, n_kv_heads=4, head_dim=128, rank=16, top_k=3,
                context=3000, dtype="bf16", seed=21, span_min=16, span_max=200),
        _custom("g8-f32-d64-r64", n_q_heads=16, n_kv_heads=2, head_dim=64, rank=64, top_k=5,
                context=5000, dtype="f32", seed=22, span_min=40, span_max=300, variant="N"),
        _custom("g2-bf16-d64-r32-ragged", batch=4, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=32,
                top_k=6, context=4000, n_prefix_anchors=40, window=64, dtype="bf16", seed=23,
                span_min=8, span_max=520, ragged=True, variant="N"),
        _custom("g4-f32-d128-r8-k1", batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=8,
                top_k=1, context=2500, dtype="f32", seed=24, span_min=16, span_max=64),
        _custom("k0-bf16", batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16, top_k=0,
                context=2000, dtype="bf16", seed=25, span_min=32, span_max=128),
        _custom("k-exceeds-spans", batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8,
                top_k=64, context=600, n_prefix_anchors=0, window=0, dtype="f32", seed=26,
                span_min=16, span_max=64),
        _custom("long-spans-multiblock", batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128,
                rank=32, top_k=4, context=12000, dtype="bf16", seed=27, span_min=600,
                span_max=1500, variant="N"),
        _custom("many-spans-merge-rounds", batch=1, n_q_heads=4, n_kv_heads=1, head_dim=64,
                rank=8, top_k=64, context=70000, dtype="bf16", seed=28, span_min=8, span_max=16),
        # many (sequence, KV head) pairs: each share item zooms several selection slots
        # (128 pairs -> 4 items per pair for k = 7; 160 pairs -> 4 items for k = 9)
        _custom("multi-slot-bf16-k7-ragged", batch=16, n_q_heads=16, n_kv_heads=8, head_dim=64,
                rank=16, top_k=7, context=2000, n_prefix_anchors=32, window=64, dtype="bf16",
                seed=29, span_min=16, span_max=160, ragged=True, variant="N"),
        _custom("multi-slot-f32-k9", batch=40, n_q_heads=8, n_kv_heads=4, head_dim=64, rank=8,
                top_k=9, context=1200, n_prefix_anchors=16, window=32, dtype="f32", seed=30,
                span_min=16, span_max=96),
        # 256 pairs x 2 routing chunks fill a whole round of routing items, so every share
        # item starts after one; two share items per pair zoom ranks {0, 2, 4} and {1, 3}
        _custom("full-route-round-bf16-k5", batch=32, n_q_heads=16, n_kv_heads=8, head_dim=64,
                rank=16, top_k=5, context=3500, n_prefix_anchors=32, window=64, dtype="bf16",
                seed=33, span_min=16, span_max=32, variant="N"),
        # the 32-layer workload's shape of work: 256 pairs x 2 routing chunks, two share
        # items per pair with four spans each at rank 16 and up to 392 anchors each (three
        # full anchor blocks and a partial one); ragged: a sequence without spans, one
        # without anchors, one with few spans, one with a third of its anchors
        _custom("many-anchors-multi-span-bf16-k8-ragged", batch=32, n_q_heads=32, n_kv_heads=8,
                head_dim=128, rank=16, top_k=8, context=4000, n_prefix_anchors=256, window=512,
                dtype="bf16", seed=34, span_min=16, span_max=32, ragged=True, variant="N"),
        # float32, three share items per pair (three spans, then two); the first round ends
        # inside the share items, so the first slot folds all 768+ anchors (seven blocks)
        _custom("many-anchors-multi-span-f32-k7", batch=24, n_q_heads=8, n_kv_heads=8,
                head_dim=64, rank=16, top_k=7, context=2000, n_prefix_anchors=256, window=512,
                dtype="f32", seed=35, span_min=24, span_max=120),
        # rank 32 with four spans per share item and many anchors
        _custom("many-anchors-multi-span-bf16-r32-k8", batch=32, n_q_heads=16, n_kv_heads=8,
                head_dim=64, rank=32, top_k=8, context=2500, n_prefix_anchors=256, window=512,
                dtype="bf16", seed=36, span_min=32, span_max=200),
    ]
    return out


CASES = small_cases()


@pytest.mark.parametrize("name,case", CASES, ids=[c[0] for c in CASES])
def test_decode_step_matches_oracle(S, name, case):
    import torch
    banner(f"decode_step {name}")
    ref = oracle_result(case)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    out_dtypes = [case.dtype] + (["f32"] if case.dtype == "bf16" else [])
    for od in out_dtypes:
        dims = dims_for(S, case, out_dtype=od)
        ws = S.Workspace(dims, dev)
        sel, out = S.decode_step(dims, dc, ws)
        torch.cuda.synchronize()
        assert ws.status() == 0
        got_sel = sel.cpu().numpy()
        if not np.array_equal(got_sel, ref["sel"]):
            bad = np.argwhere(got_sel != ref["sel"])[:5]
            raise AssertionError(f"{name}: selection differs at {bad.tolist()}; "
                                 f"min boundary gap {min_boundary_gap(ref, case):.3e}")
        assert_out_close(out_to_f64(out), ref["out"], od, where=f"{name} out={od}")
        # bitwise determinism across launches (the workspace is reused as-is)
        sel2, out2 = S.decode_step(dims, dc, ws)
        torch.cuda.synchronize()
        assert torch.equal(sel, sel2) and torch.equal(out.view(torch.uint8) if out.dtype == torch.bfloat16
                                                      else out, out2.view(torch.uint8)
                                                      if out2.dtype == torch.bfloat16 else out2)
        assert ws.status() == 0


@pytest.mark.parametrize("name,case", CASES, ids=[c[0] for c in CASES])
def test_route_then_attend_matches_oracle(S, name, case):
    import torch
    banner(f"route_topk + zoom_attend {name}")
    ref = oracle_result(case)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel, logits = S.route_topk(dims, dc, ws)
    torch.cuda.synchronize()
    assert np.array_equal(sel.cpu().numpy(), ref["sel"]), f"{name}: route_topk selection differs"
    lg = logits.cpu().numpy().astype(np.float64)
    rl = ref["logits"]
    fin = np.isfinite(rl)
    assert np.array_equal(np.isfinite(lg), fin)
    if fin.any():
        assert np.max(np.abs(lg[fin] - rl[fin]) / np.maximum(np.abs(rl[fin]), 1e-30)) <= 2 ** -23
    for given in (logits, None):
        out = S.zoom_attend(dims, dc, sel, given, ws)
        torch.cuda.synchronize()
        assert_out_close(out_to_f64(out), ref["out"], case.dtype,
                         where=f"{name} zoom_attend logits={'given' if given is not None else 'recomputed'}")
    assert ws.status() == 0


def test_workspace_reuse_across_shapes(S):
    """One workspace serves calls of different sizes back to back (counters self-reset)."""
    import torch
    dev = torch.device("cuda:0")
    big = make_case(custom_spec(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16, top_k=4,
                                context=6000, dtype="bf16", seed=31, span_min=32, span_max=256))
    small = make_case(custom_spec(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16,
                                  top_k=2, context=1500, dtype="bf16", seed=32, span_min=32,
                                  span_max=256))
    dims_big = dims_for(S, big)
    ws = S.Workspace(dims_big, dev)
    for case in (big, small, big):
        ref = oracle_result(case)
        dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
        sel, out = S.decode_step(dims_for(S, case), dc, ws)
        torch.cuda.synchronize()
        assert np.array_equal(sel.cpu().numpy(), ref["sel"])
        assert_out_close(out_to_f64(out), ref["out"], case.dtype)
    assert ws.status() == 0


def test_workspace_reuse_few_then_many_pairs(S):
    """One workspace, calls alternating between 2 and 160 (sequence, KV head) pairs: the
    second layout's counters and tagged words lie where the first layout kept other data,
    so the library must re-zero the workspace when the layout changes."""
    import torch
    dev = torch.device("cuda:0")
    few = make_case(custom_spec(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=64, rank=16, top_k=2,
                                context=1500, dtype="bf16", seed=35, span_min=16, span_max=64))
    many = make_case(custom_spec(batch=40, n_q_heads=8, n_kv_heads=4, head_dim=64, rank=16,
                                 top_k=9, context=1200, n_prefix_anchors=16, window=32,
                                 dtype="bf16", seed=36, span_min=16, span_max=96), variant="N")
    nbytes = max(S.workspace_size(dims_for(S, few)), S.workspace_size(dims_for(S, many)))
    ws = S.Workspace(dims_for(S, many), dev, nbytes=nbytes)
    refs = {id(c): oracle_result(c) for c in (few, many)}
    dcs = {id(c): S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev) for c in (few, many)}
    for i, case in enumerate((few, many, few, many, many, few)):
        banner(f"workspace reuse: call {i}, {case.spec.batch * case.spec.n_kv_heads} pairs")
        ref = refs[id(case)]
        sel, out = S.decode_step(dims_for(S, case), dcs[id(case)], ws)
        torch.cuda.synchronize()
        assert ws.status() == 0, f"call {i}"
        assert np.array_equal(sel.cpu().numpy(), ref["sel"]), f"call {i}: selection differs"
        assert_out_close(out_to_f64(out), ref["out"], case.dtype, where=f"call {i}")


def test_step_completes_while_another_stream_holds_the_device(S):
    """A decode step launched while matrix products on a second stream (same priority)
    hold compute units: work items are claimed in order, so the step's waits end and
    its results are exact, whatever the residency."""
    import torch
    banner("concurrent: decode_step beside matmuls on a second stream")
    dev = torch.device("cuda:0")
    case = make_case(WORKLOADS["llama3-8b-layer-32k"], variant="N")
    ref = oracle_result(case)
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    a = torch.randn(4096, 4096, device=dev, dtype=torch.bfloat16)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(side):
            for _ in range(8):
                b = a @ a
        sel, out = S.decode_step(dims, dc, ws)
        torch.cuda.synchronize()
        assert ws.status() == 0, f"rep {rep}: a wait timed out"
        assert np.array_equal(sel.cpu().numpy(), ref["sel"]), f"rep {rep}: selection differs"
        assert_out_close(out_to_f64(out), ref["out"], case.dtype, where=f"concurrent rep {rep}")
    del b


# One small case per kernel instantiation (storage type x head_dim x group size), so every
# compiled variant of the step kernel is checked against the oracle.
INSTANTIATIONS = [(dt, d, g) for dt in ("bf16", "f32") for d in (64, 128) for g in (1, 2, 4, 8)]


@pytest.mark.parametrize("dtype,head_dim,group", INSTANTIATIONS,
                         ids=[f"{dt}-d{d}-g{g}" for dt, d, g in INSTANTIATIONS])
def test_every_kernel_instantiation(S, dtype, head_dim, group):
    import torch
    banner(f"instantiation {dtype} d{head_dim} G{group}")
    n_kv = 2
    case = make_case(custom_spec(batch=2, n_q_heads=n_kv * group, n_kv_heads=n_kv,
                                 head_dim=head_dim, rank=16, top_k=3, context=1800,
                                 n_prefix_anchors=24, window=64, dtype=dtype,
                                 seed=40 + 8 * (dtype == "f32") + 2 * (head_dim == 128) + group,
                                 span_min=16, span_max=200), variant="N")
    ref = oracle_result(case)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel, out = S.decode_step(dims, dc, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel.cpu().numpy(), ref["sel"]), \
        f"selection differs; min boundary gap {min_boundary_gap(ref, case):.3e}"
    assert_out_close(out_to_f64(out), ref["out"], case.dtype,
                     where=f"{dtype} d{head_dim} G{group}")


def test_block_outside_arena_is_skipped_and_flagged(S):
    """A selected span whose block offset points past the factor arena: the kernels do
    not read it (no fault), set the block-range bit of the error word, keep the
    selection, and leave every other (sequence, KV head) pair's output bit for bit."""
    import torch
    banner("block outside the arena: fused step and route + attend")
    dev = torch.device("cuda:0")
    case = make_case(custom_spec(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=64, rank=16,
                                 top_k=3, context=2500, dtype="bf16", seed=34, span_min=32,
                                 span_max=160), variant="N")
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    sel0, out0 = S.decode_step(dims, dc, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    sel0 = sel0.cpu().numpy()
    out0 = out0.cpu()
    bad = case_arrays(case)
    bad["block_off"] = case.block_off.copy()
    s_bad = int(sel0[0, 0, 0])                           # the best span of (b 0, KV head 0)
    bad["block_off"][0, 0, s_bad] = case.factors.nbytes  # one byte past the end of the arena
    dcb = S.DeviceCache.from_arrays(bad, case.dtype, dev)
    G = case.spec.n_q_heads // case.spec.n_kv_heads
    for how in ("fused", "route+attend"):
        if how == "fused":
            sel, out = S.decode_step(dims, dcb, ws)
        else:
            sel, logits = S.route_topk(dims, dcb, ws)
            out = S.zoom_attend(dims, dcb, sel, logits, ws)
        torch.cuda.synchronize()
        assert ws.status() & 2, f"{how}: block-range bit not set"
        assert np.array_equal(sel.cpu().numpy(), sel0), f"{how}: selection changed"
        o = out.cpu()
        assert torch.equal(o[0, G:], out0[0, G:]) and torch.equal(o[1], out0[1]), \
            f"{how}: an unaffected pair's output changed"
        assert not torch.equal(o[0, :G], out0[0, :G]), f"{how}: the skipped span changed nothing"


@pytest.mark.parametrize("variant", ["L", "N"])
def test_layer_128k_b4_full_size(S, variant):
    """The 128K-context, batch-4 layer at full size: every selection and every output row."""
    import torch
    banner(f"128K x 4 full size, variant {variant}: generating")
    case = make_case(WORKLOADS["llama3-8b-layer-128k-b4"], variant=variant)
    banner("128K x 4: oracle")
    ref = oracle_result(case)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    banner("128K x 4: decode_step")
    sel, out = S.decode_step(dims, dc, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel.cpu().numpy(), ref["sel"]), \
        f"selection differs; min boundary gap {min_boundary_gap(ref, case):.3e}"
    assert_out_close(out_to_f64(out), ref["out"], "bf16", where=f"128K x 4 {variant}")
    # the launch configuration the bench times: graph replays over cache copies, each
    # node the same kernel on its own copy; every node must give the stream launch's bits
    banner("128K x 4: graph replays over two cache copies")
    copy = S.DeviceCache({k: v.clone() for k, v in dc.t.items()}, case.dtype)
    g = S.LayerGraph(dims, [dc, copy], ws)
    try:
        for _ in range(3):
            gsel, gout = g.launch()
            torch.cuda.synchronize()
            assert ws.status() == 0
            for l in range(2):
                assert torch.equal(gsel[l], sel), f"graph node {l}: selection differs"
                assert torch.equal(gout[l], out), f"graph node {l}: output differs"
    finally:
        g.destroy()
