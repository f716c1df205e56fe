"""GPU: sekv_decode_step_noalloc (workspace in the library's static device array) against
sekv_decode_step on a caller workspace: two calls in a row, the second with a smaller
input, and a call whose shapes need more than the array holds (refused)."""

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


def _same(a, b):
    import torch
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a, b)


def test_noalloc_matches_decode_step_twice_then_smaller(S):
    import torch
    dev = torch.device("cuda:0")
    big = make_case(WORKLOADS["llama3-8b-layer-32k"], variant="N")
    small = make_case(custom_spec(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, rank=16,
                                  top_k=3, context=2500, dtype="bf16", seed=81, span_min=16,
                                  span_max=128), variant="N")
    for i, case in enumerate((big, big, small)):
        banner(f"noalloc call {i}: batch {case.spec.batch}, {int(case.n_spans.max())} spans")
        dims = dims_for(S, case)
        dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
        ws = S.Workspace(dims, dev)
        sel_ref, out_ref = S.decode_step(dims, dc, ws)
        sel, out = S.decode_step_noalloc(dims, dc)
        torch.cuda.synchronize()
        assert ws.status() == 0
        assert torch.equal(sel, sel_ref), f"call {i}: selection differs from sekv_decode_step"
        assert _same(out, out_ref), f"call {i}: output differs from sekv_decode_step"
        ref = oracle_result(case)
        assert np.array_equal(sel.cpu().numpy(), ref["sel"]), f"call {i}: selection differs from the oracle"
        assert_out_close(out_to_f64(out), ref["out"], case.dtype, where=f"noalloc call {i}")


def test_noalloc_refuses_shapes_beyond_its_array(S):
    import torch
    dev = torch.device("cuda:0")
    case = make_case(custom_spec(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=64, rank=8, top_k=2,
                                 context=600, dtype="f32", seed=82))
    dims = dims_for(S, case)
    dims.batch = 4096                      # about 4096 x 2 pairs of partials: past 16 MiB
    dims.max_spans = 512
    assert S.workspace_size(dims) > S.NOALLOC_MAX_WORKSPACE
    dc = S.DeviceCache.from_arrays(case_arrays(case), case.dtype, dev)
    with pytest.raises(S.SekvError) as ei:
        S.decode_step_noalloc(dims, dc, sel=torch.empty(1, dtype=torch.int32, device=dev),
                              out=torch.empty(1, dtype=torch.float32, device=dev))
    assert ei.value.status == S.SEKV_ERR_WORKSPACE and "noalloc" in str(ei.value)
