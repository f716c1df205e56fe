"""The C-ABI library on the CPU: it loads, exports every declared symbol, and rejects
bad arguments on the host before touching the GPU."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sekv.h")
LIB = os.path.join(ROOT, "paper_2606_31145_amd", "libsekv.so")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SEKV_API\s+[\w\s\*]*?\b(sekv_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def S():
    if not os.path.exists(LIB):
        from paper_2606_31145_amd.build import build
        build()
    from paper_2606_31145_amd import sekv
    return sekv


def test_header_declares_the_boundary():
    names = declared_functions()
    for fn in ("sekv_route_topk", "sekv_zoom_attend", "sekv_decode_step", "sekv_workspace_size"):
        assert fn in names


def test_library_exports_every_declared_symbol(S):
    lib = ctypes.CDLL(LIB)
    for fn in declared_functions():
        assert hasattr(lib, fn), f"{fn} declared in sekv.h but not exported"
    assert set(declared_functions()) == set(S.EXPORTED)


def _dims(S, **kw):
    base = dict(batch=1, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8, top_k=2, max_anchors=33,
                max_spans=49, max_span_len=64, dtype="f32", softmax_scale=0.125)
    base.update(kw)
    return S.make_dims(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(n_q_heads=6, n_kv_heads=4), 1),          # Hq % Hkv
    (dict(n_q_heads=12, n_kv_heads=4), 2),         # group 3
    (dict(head_dim=96), 2),
    (dict(rank=12), 2),
    (dict(rank=24), 2),
    (dict(rank=72), 2),
    (dict(top_k=65), 2),
    (dict(max_spans=0), 1),
    (dict(max_span_len=0), 1),
    (dict(batch=-1), 1),
    (dict(softmax_scale=0.0), 1),
    (dict(dtype="f32", out_dtype="bf16"), 2),
    (dict(max_spans=80000), 2),                    # too many partials per pair
])
def test_check_dims_rejects(S, kw, status):
    d = _dims(S, **kw)
    with pytest.raises(S.SekvError) as ei:
        S.check_dims(d)
    assert ei.value.status == status
    assert S.workspace_size(d) == 0


def test_check_dims_accepts_the_workload_shapes(S):
    S.check_dims(_dims(S))
    big = _dims(S, batch=4, n_q_heads=32, n_kv_heads=8, head_dim=128, rank=32, top_k=16,
                max_anchors=800, max_spans=760, max_span_len=512, dtype="bf16",
                softmax_scale=128 ** -0.5)
    S.check_dims(big)
    assert S.workspace_size(big) > 0


def test_host_errors_before_any_launch(S):
    """Null pointers and a short workspace are rejected without a HIP call."""
    d = _dims(S)
    cache = S.CacheStruct()              # all NULL
    st = S.LIB.sekv_decode_step(ctypes.byref(d), ctypes.byref(cache), None, None, None, 0, None)
    assert st == S.SEKV_ERR_INVALID_ARG
    assert b"NULL" in S.LIB.sekv_last_error()
    fake = ctypes.c_void_p(0x10000)      # aligned, never dereferenced on the host path below
    c2 = S.CacheStruct(*([0x10000] * 10), 4096, 0x10000)
    st = S.LIB.sekv_decode_step(ctypes.byref(d), ctypes.byref(c2), fake, fake, fake, 16, None)
    assert st == S.SEKV_ERR_WORKSPACE
    c3 = S.CacheStruct(0x10008, *([0x10000] * 9), 4096, 0x10000)
    st = S.LIB.sekv_route_topk(ctypes.byref(d), ctypes.byref(c3), fake, None, fake, 1 << 20, None)
    assert st == S.SEKV_ERR_INVALID_ARG and b"aligned" in S.LIB.sekv_last_error()
    assert S.LIB.sekv_status_string(3) == b"SEKV_ERR_WORKSPACE"


def test_empty_batch_is_a_no_op(S):
    d = _dims(S, batch=0)
    c = S.CacheStruct()
    fake = ctypes.c_void_p(0x10000)
    ws = S.workspace_size(d)
    assert S.LIB.sekv_decode_step(ctypes.byref(d), ctypes.byref(c), None, None, fake, ws, None) == 0


def test_validate_cache_on_host_copies(S):
    """sekv_validate_cache checks the device-side preconditions on host copies."""
    import numpy as np

    from synth import custom_spec, make_case
    case = make_case(custom_spec(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8,
                                 top_k=2, context=900, dtype="bf16", seed=71))
    arrays = dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v,
                  n_anchors=case.n_anchors, sum_k=case.sum_k, sum_v=case.sum_v,
                  n_spans=case.n_spans, span_len=case.span_len, span_logsize=case.span_logsize,
                  factors=case.factors, block_off=case.block_off)
    d = _dims(S, **{k: v for k, v in case.dims().items()})
    S.validate_cache(d, arrays)

    def bad(field, fn, msg):
        a = dict(arrays)
        a[field] = np.array(arrays[field], copy=True)
        fn(a[field])
        with pytest.raises(S.SekvError) as ei:
            S.validate_cache(d, a)
        assert ei.value.status == S.SEKV_ERR_INVALID_ARG and msg in str(ei.value), str(ei.value)

    bad("n_spans", lambda x: x.__setitem__(0, case.max_spans + 1), "n_spans")
    bad("n_anchors", lambda x: x.__setitem__(1, -1), "n_anchors")
    bad("span_len", lambda x: x.__setitem__((0, 0), 0), "span_len")
    bad("span_logsize", lambda x: x.__setitem__((1, 2), 9.0), "span_logsize")
    bad("block_off", lambda x: x.__setitem__((1, 1, 0), case.factors.nbytes), "outside")
    bad("q", lambda x: x.__setitem__((0, 1, 3), 0x7FC0), "not finite")        # bf16 NaN
    bad("sum_v", lambda x: x.__setitem__((1, 0, 0, 5), 0x7F80), "not finite")  # bf16 +inf


def test_validate_cache_adaptive_ranks(S):
    """Per-block ranks: a valid ragged-rank cache passes; a rank off the 16-byte granule,
    above the common rank, or a block that no longer fits the arena fails."""
    import numpy as np

    from synth import custom_spec, make_case
    case = make_case(custom_spec(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=16, top_k=2,
                                 context=900, dtype="bf16", seed=72, rank_mode="adaptive"))
    arrays = dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v,
                  n_anchors=case.n_anchors, sum_k=case.sum_k, sum_v=case.sum_v,
                  n_spans=case.n_spans, span_len=case.span_len, span_logsize=case.span_logsize,
                  factors=case.factors, block_off=case.block_off, block_rank=case.block_rank)
    d = _dims(S, **{k: v for k, v in case.dims().items()})
    S.validate_cache(d, arrays)
    for word, msg in ((4 | (8 << 16), "ranks"), (24 | (8 << 16), "ranks"), (16 | (0 << 16), "ranks")):
        a = dict(arrays, block_rank=case.block_rank.copy())
        a["block_rank"][0, 1, 2] = word
        with pytest.raises(S.SekvError) as ei:
            S.validate_cache(d, a)
        assert msg in str(ei.value), str(ei.value)
    # the last block of the arena grown to the full rank no longer fits
    last = np.unravel_index(np.argmax(case.block_off), case.block_off.shape)
    a = dict(arrays, block_rank=case.block_rank.copy())
    a["block_rank"][last] = 16 | (16 << 16)
    w = int(case.block_rank[last])
    if (w & 0xFFFF, w >> 16) != (16, 16):
        with pytest.raises(S.SekvError) as ei:
            S.validate_cache(d, dict(a, factors=case.factors[:int(case.block_off[last]) +
                                                             (int(case.span_len[last[0], last[2]]) + 65) *
                                                             ((w & 0xFFFF) + (w >> 16)) * 2]))
        assert "outside" in str(ei.value)


def test_layered_tier_rejects_null_arguments(S):
    """sekv_decode_layers_tiered and sekv_tier_layer_stats fail on the host, before any device
    call, without a tier or counters."""
    dims = _dims(S)
    with pytest.raises(S.SekvError):
        S._check(S.LIB.sekv_decode_layers_tiered(ctypes.byref(dims), None, None, 2, 1, None, None, None,
                                                 None, 0, None, None))
    with pytest.raises(S.SekvError):
        S._check(S.LIB.sekv_tier_layer_stats(None, None))
