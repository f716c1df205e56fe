"""GPU: the pinned-host tier (sekv_decode_step_tiered).  The factor arena lives in pinned
host memory and only the selected spans' blocks are copied to the device each step.

Checked against the same computation on a device-resident arena (sekv_route_topk, then
sekv_zoom_attend with the routing scores: bitwise) and against the CPU oracle."""

import numpy as np
import pytest

from synth import WORKLOADS, custom_spec, make_case
from synth.cases import block_bytes
from tests.gpu_common import (assert_out_close, banner, case_arrays, dims_for, oracle_result,
                              out_to_f64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


MODES = ["gather", "memcpy"]


def _tier_case(S, case, steps=2, mode="gather"):
    import torch
    dev = torch.device("cuda:0")
    dims = dims_for(S, case)
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    ws = S.Workspace(dims, dev)
    # device-resident reference: route, then attend with the routing scores
    sel_r, logits = S.route_topk(dims, dc, ws)
    out_r = S.zoom_attend(dims, dc, sel_r, logits, ws)
    torch.cuda.synchronize()
    host = S.HostFactors(case.factors, case.block_off, case.span_len)
    tier = S.Tier(dims, mode)
    side = torch.cuda.Stream()
    ref = oracle_result(case)
    try:
        for step in range(steps):
            sel, out = S.decode_step_tiered(dims, dc, host, tier, ws, side=side)
            torch.cuda.synchronize()
            assert ws.status() == 0
            assert np.array_equal(sel.cpu().numpy(), ref["sel"]), f"step {step}: selection differs"
            assert torch.equal(sel, sel_r)
            assert torch.equal(out.view(torch.uint8) if out.dtype == torch.bfloat16 else out,
                               out_r.view(torch.uint8) if out_r.dtype == torch.bfloat16 else out_r), \
                f"step {step}: output differs from the device-resident path"
            assert_out_close(out_to_f64(out), ref["out"], case.dtype, where=f"tier {mode} step {step}")
            nbytes, ncopies, ms = tier.last_copy()
            s = ref["sel"]
            lens = [int(case.span_len[b, x]) for b in range(s.shape[0]) for g in range(s.shape[1])
                    for x in s[b, g] if x >= 0]
            raw = sum(block_bytes(L, case.spec.rank, case.spec.head_dim, case.dtype) for L in lens)
            tight = sum(2 * case.spec.rank * (L + case.spec.head_dim + 1) for L in lens) * \
                (2 if case.dtype == "bf16" else 4)
            assert tight <= nbytes <= raw, (tight, nbytes, raw)
            if mode == "gather":
                assert ncopies == len(lens)          # one copy per selected block
            else:
                assert (ncopies <= len(lens)) and (ncopies > 0) == (len(lens) > 0)
            if lens:
                assert ms > 0.0
    finally:
        tier.destroy()
    return tier


@pytest.mark.parametrize("mode", MODES)
def test_tier_small_bf16(S, mode):
    banner(f"tier: small bf16, {mode}")
    spec = custom_spec(batch=3, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16, top_k=5,
                       context=4000, n_prefix_anchors=64, window=128, dtype="bf16", seed=51,
                       span_min=32, span_max=300)
    _tier_case(S, make_case(spec, variant="N"), mode=mode)


@pytest.mark.parametrize("mode", MODES)
def test_tier_small_f32_ragged(S, mode):
    banner(f"tier: small f32, ragged tables, {mode}")
    spec = custom_spec(batch=4, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8, top_k=6,
                       context=1500, n_prefix_anchors=16, window=0, dtype="f32", seed=52,
                       span_min=8, span_max=40)
    c = make_case(spec)
    c.n_spans = c.n_spans.copy()
    c.n_anchors = c.n_anchors.copy()
    c.n_spans[1] = 0
    c.n_spans[2] = 3               # fewer spans than top_k
    c.n_anchors[3] = 0
    _tier_case(S, c, mode=mode)


def test_tier_adjacent_blocks_coalesce(S):
    """k = all spans: every block of a sequence is selected, and the arena holds the
    blocks of (sequence, KV head, span) in order, so each sequence moves with one copy."""
    banner("tier: k = all spans")
    import torch
    spec = custom_spec(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8, top_k=64,
                       context=700, n_prefix_anchors=8, window=0, dtype="f32", seed=53,
                       span_min=16, span_max=40)
    c = make_case(spec)
    assert int(c.n_spans.max()) <= 64
    _tier_case(S, c, steps=1, mode="memcpy")
    dims = dims_for(S, c)
    dev = torch.device("cuda:0")
    tier = S.Tier(dims, "memcpy")
    try:
        dc = S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev)
        ws = S.Workspace(dims, dev)
        host = S.HostFactors(c.factors, c.block_off, c.span_len)
        S.decode_step_tiered(dims, dc, host, tier, ws, side=torch.cuda.Stream())
        torch.cuda.synchronize()
        _, ncopies, _ = tier.last_copy()
        # the arena holds (sequence, KV head, span) in order: one run per sequence
        assert ncopies == spec.batch
    finally:
        tier.destroy()


@pytest.mark.parametrize("variant,mode", [("L", "gather"), ("N", "gather"), ("L", "memcpy"),
                                          ("N", "memcpy")])
def test_tier_128k_b4_full_size(S, variant, mode):
    """The 128K x 4 host-tier workload at full size (literal and planted values)."""
    banner(f"tier: 128K x 4 full size, variant {variant}, {mode}: generating")
    case = make_case(WORKLOADS["llama3-8b-layer-128k-b4-hosttier"], variant=variant)
    banner("tier: 128K x 4: running")
    _tier_case(S, case, steps=2, mode=mode)


def test_tier_gather_skips_blocks_outside_the_arena(S):
    """Gather mode plans on the device: a selected block whose arena offset lies past the
    arena is skipped and flagged in the workspace error word (bit 2), with no fault."""
    import torch
    banner("tier gather: block outside the arena")
    spec = custom_spec(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=64, rank=16, top_k=3,
                       context=2500, dtype="bf16", seed=55, span_min=32, span_max=160)
    c = make_case(spec, variant="N")
    dims = dims_for(S, c)
    dev = torch.device("cuda:0")
    ref = oracle_result(c)
    bad = case_arrays(c)
    bad["block_off"] = c.block_off.copy()
    s_bad = int(ref["sel"][0, 0, 0])
    bad["block_off"][0, 0, s_bad] = c.factors.nbytes
    dc = S.DeviceCache.from_arrays(bad, c.dtype, dev)
    ws = S.Workspace(dims, dev)
    host = S.HostFactors(c.factors, bad["block_off"], c.span_len)
    tier = S.Tier(dims, "gather")
    try:
        sel, out = S.decode_step_tiered(dims, dc, host, tier, ws, side=torch.cuda.Stream())
        torch.cuda.synchronize()
        assert ws.status() & 2
        assert np.array_equal(sel.cpu().numpy(), ref["sel"])
        G = spec.n_q_heads // spec.n_kv_heads
        assert_out_close(out_to_f64(out[1]), ref["out"][1], c.dtype, where="unaffected sequence")
        assert_out_close(out_to_f64(out[0, G:]), ref["out"][0, G:], c.dtype, where="unaffected head")
    finally:
        tier.destroy()
    host_m = S.HostFactors(c.factors, bad["block_off"], c.span_len)
    tier_m = S.Tier(dims, "memcpy")
    try:
        with pytest.raises(S.SekvError) as ei:
            S.decode_step_tiered(dims, dc, host_m, tier_m, ws, side=torch.cuda.Stream())
        assert ei.value.status == S.SEKV_ERR_INVALID_ARG
        torch.cuda.synchronize()
    finally:
        tier_m.destroy()


@pytest.mark.parametrize("mode", MODES)
def test_tier_rejects_unpinned_arena(S, mode):
    import torch
    spec = custom_spec(batch=1, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8, top_k=2,
                       context=600, dtype="f32", seed=54)
    c = make_case(spec)
    dims = dims_for(S, c)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev)
    ws = S.Workspace(dims, dev)
    host = S.HostFactors(c.factors, c.block_off, c.span_len)
    host.arena = torch.from_numpy(np.ascontiguousarray(c.factors))     # pageable memory
    tier = S.Tier(dims, mode)
    try:
        with pytest.raises(S.SekvError) as ei:
            S.decode_step_tiered(dims, dc, host, tier, ws, side=torch.cuda.Stream())
        assert ei.value.status == S.SEKV_ERR_INVALID_ARG and "pinned" in str(ei.value)
    finally:
        tier.destroy()
