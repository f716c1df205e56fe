"""GPU: exact ties in the selection key resolve to the lower span index (Sec. 3.3 budget
rule read as a total order: key descending, span index ascending).

A tie is planted the way a duplicated span produces one: span T gets the summary key row
of span S (sum_k[b][g][T] = sum_k[b][g][S]) where both spans have the same length, so
every query head scores them identically, ln|S| included, and the fp64 selection keys are
equal bit for bit.  Ties are placed where each path of the selection meets them:

* both spans in one routing chunk of 128 spans and in the same 64-span sorting half;
* one chunk, opposite halves;
* different chunks;
* straddling the k-th place (one of the two is selected, the other is not);
* a pair with more than 512 candidates, which is ranked by the single-merger path.

Selections are compared bit for bit with the oracle through sekv_decode_step, through
sekv_route_topk + sekv_zoom_attend, and through the host tier.
"""

import numpy as np
import pytest

from synth import custom_spec, make_case
from tests.gpu_common import (assert_out_close, banner, case_arrays, dims_for, oracle_result,
                              out_to_f64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_31145_amd import sekv
    return sekv


def _partner(case, b, src, want, taken):
    """A span index near `want` with the length of span `src` (not `src`, not taken)."""
    m = int(case.n_spans[b])
    L = int(case.span_len[b, src])
    order = sorted(range(m), key=lambda t: (abs(t - want), t))
    for t in order:
        if t != src and t not in taken and int(case.span_len[b, t]) == L:
            return t
    raise AssertionError(f"no span of length {L} near {want}")


def _plant(case, b, g, src, dst):
    case.sum_k = case.sum_k.copy() if not case.sum_k.flags.writeable else case.sum_k
    case.sum_k[b, g, dst] = case.sum_k[b, g, src]


def _keys(case):
    """The oracle's selection keys of the case as it stands."""
    import oracle
    from synth.cases import from_storage
    s = case.spec
    lg = oracle.routing_logits(from_storage(case.q, s.dtype), from_storage(case.sum_k, s.dtype),
                               case.span_logsize, case.n_spans, s.softmax_scale)
    return oracle.group_keys(lg, s.n_kv_heads)


def _rank_order(keys_row, m):
    return sorted(range(m), key=lambda t: (-keys_row[t], t))


def _tie_case(seed, k, context, span_min, span_max, batch=2, n_kv=2, group=4, head_dim=64,
              rank=8, dtype="bf16", placements=("same-half", "opposite-half", "other-chunk",
                                                "boundary")):
    """A case with exact ties planted in every (b, g) pair at the given placements."""
    case = make_case(custom_spec(batch=batch, n_q_heads=n_kv * group, n_kv_heads=n_kv,
                                 head_dim=head_dim, rank=rank, top_k=k, context=context,
                                 n_prefix_anchors=16, window=32, dtype=dtype, seed=seed,
                                 span_min=span_min, span_max=span_max))
    case.sum_k = case.sum_k.copy()
    planted = []
    for b in range(batch):
        m = int(case.n_spans[b])
        for g in range(n_kv):
            taken = set()
            for what in placements:
                # the order as planted so far (later ties shift the k-th place)
                order = _rank_order(_keys(case)[b, g], m)
                if what == "boundary":
                    src = order[min(k, m) - 1]          # the k-th best span
                    want = src + 37
                else:
                    src = next(t for t in order if t not in taken)   # a span near the top
                    base = (src // 128) * 128
                    half = (src % 128) // 64
                    if what == "same-half":
                        want = base + 64 * half + (src % 64 + 23) % 64
                    elif what == "opposite-half":
                        want = base + 64 * (1 - half) + src % 64
                    else:
                        want = (src + 300) % max(m, 1)
                dst = _partner(case, b, src, want, taken)
                _plant(case, b, g, src, dst)
                taken |= {src, dst}
                planted.append((b, g, what, src, dst))
    return case, planted


def _check_ties_resolved(ref, case, planted):
    """The oracle itself: every planted pair ties exactly, and the lower index ranks first."""
    keys = ref["keys"]
    seen_boundary = False
    for b, g, what, src, dst in planted:
        assert keys[b, g, src] == keys[b, g, dst], (b, g, what, src, dst)
        sel = list(ref["sel"][b, g])
        lo, hi = min(src, dst), max(src, dst)
        if hi in sel:
            assert lo in sel and sel.index(lo) < sel.index(hi), (b, g, what, sel)
        if what == "boundary" and (lo in sel) != (hi in sel):
            seen_boundary = True
    return seen_boundary


CASES = [
    # m about 2 * 128 spans: ties inside one chunk (both halves) and across chunks
    dict(seed=61, k=6, context=9000, span_min=16, span_max=40),
    # a single routing chunk per pair
    dict(seed=62, k=4, context=2600, span_min=16, span_max=24, placements=("same-half", "opposite-half", "boundary")),
    # k = 1: the tie decides the only slot
    dict(seed=63, k=1, context=5000, span_min=16, span_max=20, placements=("boundary",)),
    # float32 storage, group 8
    dict(seed=64, k=5, context=6000, span_min=16, span_max=30, dtype="f32", group=8, head_dim=128, rank=16),
]


@pytest.mark.parametrize("kw", CASES, ids=[f"seed{c['seed']}-k{c['k']}" for c in CASES])
def test_ties_go_to_the_lower_index(S, kw):
    import torch
    kw = dict(kw)
    case, planted = _tie_case(**kw)
    banner(f"ties seed {kw['seed']}: {len(planted)} planted pairs")
    ref = oracle_result(case)
    assert _check_ties_resolved(ref, case, planted) or kw["k"] == 0
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel, out = S.decode_step(dims, dc, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel.cpu().numpy(), ref["sel"]), "decode_step: tie resolved differently"
    assert_out_close(out_to_f64(out), ref["out"], case.dtype, where="decode_step ties")
    sel2, logits = S.route_topk(dims, dc, ws)
    out2 = S.zoom_attend(dims, dc, sel2, logits, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel2.cpu().numpy(), ref["sel"]), "route_topk: tie resolved differently"
    assert_out_close(out_to_f64(out2), ref["out"], case.dtype, where="route+attend ties")
    host = S.HostFactors(case.factors, case.block_off, case.span_len)
    tier = S.Tier(dims)
    try:
        sel3, out3 = S.decode_step_tiered(dims, dc, host, tier, ws, side=torch.cuda.Stream())
        torch.cuda.synchronize()
        assert ws.status() == 0
        assert np.array_equal(sel3.cpu().numpy(), ref["sel"]), "tier: tie resolved differently"
        assert torch.equal(out3.view(torch.uint8) if out3.dtype == torch.bfloat16 else out3,
                           out2.view(torch.uint8) if out2.dtype == torch.bfloat16 else out2)
    finally:
        tier.destroy()


def test_ties_in_the_merger_path(S):
    """More than 512 candidates per pair (k = 64 over about 1 100 spans: 9 routing chunks x
    64 candidates): the single-merger path ranks them; ties planted near the top and at
    the 64th place."""
    import torch
    case, planted = _tie_case(seed=65, k=64, context=17000, span_min=12, span_max=16, batch=1,
                              n_kv=2, group=2, placements=("same-half", "opposite-half",
                                                           "other-chunk", "boundary"))
    assert int(case.n_spans.max()) > 1024
    banner(f"ties, merger path: {len(planted)} planted pairs, m = {int(case.n_spans.max())}")
    ref = oracle_result(case)
    assert _check_ties_resolved(ref, case, planted)
    dev = torch.device("cuda:0")
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    dims = dims_for(S, case)
    ws = S.Workspace(dims, dev)
    sel, out = S.decode_step(dims, dc, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    assert np.array_equal(sel.cpu().numpy(), ref["sel"]), "merger path: tie resolved differently"
    assert_out_close(out_to_f64(out), ref["out"], case.dtype, where="merger ties")
    sel2, _ = S.route_topk(dims, dc, ws)
    torch.cuda.synchronize()
    assert np.array_equal(sel2.cpu().numpy(), ref["sel"])
