"""GPU: several layers of one decode step with the factors in pinned host memory and the
cross-layer prefetch of the paper's pipelined transfer (Sec. 3.2, last paragraph):
sekv_decode_layers_tiered with and without prefetch, against each layer's route + attend
on a device-resident arena (bitwise) and the CPU oracle; the copy counters against the
selections (blocks prefetched = the previous layer's selected blocks; blocks copied after
a selection = the selected blocks the previous layer did not select)."""

import numpy as np
import pytest

from synth import custom_spec, make_case
from tests.gpu_common import assert_out_close, banner, case_arrays, dims_for, oracle_result, out_to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


def _run(S, spec, n_layers, variant="N", shared=True):
    import torch
    dev = torch.device("cuda:0")
    cases = [make_case(spec, layer=l, variant=variant, needle_layer=0 if shared else None)
             for l in range(n_layers)]
    dims = dims_for(S, cases[0])
    for c in cases[1:]:
        assert (c.max_anchors, c.max_spans, c.max_span_len) == (cases[0].max_anchors, cases[0].max_spans,
                                                                cases[0].max_span_len)
    ws = S.Workspace(dims, dev)
    dcs = [S.DeviceCache.from_arrays(case_arrays(c), c.dtype, dev) for c in cases]
    refs = []
    for dc in dcs:
        sel_r, logits = S.route_topk(dims, dc, ws)
        out_r = S.zoom_attend(dims, dc, sel_r, logits, ws)
        refs.append((sel_r.clone(), out_r.clone()))
    torch.cuda.synchronize()
    hosts = [S.HostFactors(c.factors, c.block_off, c.span_len, block_rank=c.block_rank) for c in cases]
    tier = S.Tier(dims, "gather")
    side = torch.cuda.Stream()
    k = spec.top_k
    try:
        stats = {}
        for prefetch in (False, True, True):
            sel, out = S.decode_layers_tiered(dims, dcs, hosts, tier, ws, prefetch=prefetch, side=side)
            torch.cuda.synchronize()
            assert ws.status() == 0
            for l in range(n_layers):
                assert torch.equal(sel[l], refs[l][0]), f"layer {l}: selection differs (prefetch {prefetch})"
                o, r = out[l], refs[l][1]
                if o.dtype == torch.bfloat16:
                    o, r = o.view(torch.int16), r.view(torch.int16)
                assert torch.equal(o, r), f"layer {l}: output differs (prefetch {prefetch})"
            stats[prefetch] = tier.layer_stats()
        ref0 = oracle_result(cases[0])
        assert np.array_equal(refs[0][0].cpu().numpy(), ref0["sel"])
        assert_out_close(out_to_f64(refs[0][1]), ref0["out"], cases[0].dtype, "layer 0 reference")
    finally:
        tier.destroy()
    sels = [r[0].cpu().numpy() for r in refs]
    n_sel = [int((s >= 0).sum()) for s in sels]
    hits = 0
    for l in range(1, n_layers):
        for b in range(spec.batch):
            for g in range(spec.n_kv_heads):
                prev = set(int(x) for x in sels[l - 1][b, g] if x >= 0)
                hits += sum(1 for x in sels[l][b, g] if x >= 0 and int(x) in prev)
    crit_bytes, crit_blocks, pf_bytes, pf_blocks = stats[True]
    assert stats[False][1] == sum(n_sel) and stats[False][2:] == (0, 0)
    assert pf_blocks == sum(n_sel[:-1])
    assert crit_blocks == sum(n_sel) - hits
    assert crit_bytes < stats[False][0] or hits == 0
    banner(f"layers {n_layers}: {hits} prefetch hits of {sum(n_sel[1:])} selections after the first layer; "
           f"critical bytes {crit_bytes} vs {stats[False][0]} without prefetch")
    return hits


def test_layers_tiered_bf16_shared_needles(S):
    banner("layered tier: bf16, planted spans shared by the layers")
    spec = custom_spec(batch=3, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16, top_k=6,
                       context=4000, n_prefix_anchors=64, window=128, dtype="bf16", seed=57,
                       span_min=32, span_max=300)
    hits = _run(S, spec, 3)
    assert hits > 0


def test_layers_tiered_f32_independent_layers(S):
    banner("layered tier: f32, independent layers, ragged ranks")
    spec = custom_spec(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=16, top_k=4,
                       context=2500, n_prefix_anchors=16, window=32, dtype="f32", seed=58,
                       span_min=8, span_max=120, rank_mode="adaptive")
    _run(S, spec, 4, variant="L", shared=False)


@pytest.mark.parametrize("top_k,n_layers", [(3, 1), (0, 2)])
def test_layers_tiered_one_layer_and_no_zoom(S, top_k, n_layers):
    banner(f"layered tier: k = {top_k}, {n_layers} layer(s)")
    spec = custom_spec(batch=2, n_q_heads=4, n_kv_heads=1, head_dim=64, rank=8, top_k=top_k,
                       context=1200, n_prefix_anchors=16, window=16, dtype="bf16", seed=59,
                       span_min=8, span_max=80)
    _run(S, spec, n_layers)
