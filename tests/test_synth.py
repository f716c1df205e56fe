"""The synthetic cache generator: partitions, storage rounding, determinism, planting."""

import math

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, custom_spec, make_case
from synth.cases import (bf16_bits_to_f64, f64_to_bf16_bits, from_storage, span_lengths,
                         uniforms)
from tests.helpers import oracle_kwargs


@pytest.mark.parametrize("name", ["tiny-f32", "llama3-8b-layer-32k", "llama3-8b-layer-128k-b4",
                                  "llama3-8b-32layer-32k-b32"])
def test_partition_covers_context(name):
    spec = WORKLOADS[name]
    for b in range(min(spec.batch, 4)):
        lens, rem = span_lengths(spec, b)
        assert all(spec.span_min <= L <= spec.span_max for L in lens)
        assert 0 <= rem < spec.span_min
        assert sum(lens) + rem + spec.n_prefix_anchors + spec.window == spec.context


def test_loguniform_partition_statistics():
    spec = WORKLOADS["llama3-8b-layer-128k-b4"]
    lens = [L for b in range(4) for L in span_lengths(spec, b)[0]]
    assert 165 < np.mean(lens) < 185          # E[min(512, floor(e^U))] ~ 173
    assert 680 < len(lens) / 4 < 800          # about 700 spans per 128K sequence


def test_bf16_rounding_is_nearest_even():
    g = np.random.default_rng(0)
    x = g.standard_normal(200_000) * 10.0 ** g.integers(-20, 20, 200_000)
    b = f64_to_bf16_bits(x)
    y = bf16_bits_to_f64(b)
    up, dn = bf16_bits_to_f64(b + 1), bf16_bits_to_f64(b - 1)
    assert np.all(np.abs(y - x) <= np.abs(up - x))
    assert np.all(np.abs(y - x) <= np.abs(dn - x))
    # exact halfway cases go to the even pattern
    base = bf16_bits_to_f64(np.arange(0x3F80, 0x3F90, dtype=np.uint16))
    mid = (base[:-1] + base[1:]) / 2
    got = f64_to_bf16_bits(mid)
    assert np.all(got % 2 == 0)


def test_generation_is_deterministic_and_thread_independent():
    spec = custom_spec(dtype="bf16", batch=2, n_q_heads=8, n_kv_heads=2, head_dim=64, rank=16,
                       top_k=4, context=3000, seed=5)
    a = make_case(spec, variant="N", threads=1)
    b = make_case(spec, variant="N", threads=4)
    for name in ("q", "anchor_k", "anchor_v", "sum_k", "sum_v", "factors", "block_off",
                 "span_len", "span_logsize", "needles"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    c = make_case(spec, layer=1)
    assert not np.array_equal(a.q, c.q)
    assert np.array_equal(a.span_len, c.span_len)     # partition shared across layers


def test_counter_stream_is_position_addressable():
    full = uniforms(1234, 5000)
    assert np.array_equal(full[:10], uniforms(1234, 10))
    assert 0.0 <= full.min() and full.max() < 1.0
    assert abs(full.mean() - 0.5) < 0.02


def test_tiny_config_factors_are_orthonormal():
    case = make_case(WORKLOADS["tiny-f32"])
    s = case.spec
    for S in range(int(case.n_spans[0])):
        f = oracle.read_span_block(case.factors, int(case.block_off[0, 1, S]),
                                   int(case.span_len[0, S]), s.rank, s.head_dim, s.dtype)
        for side in "KV":
            U, Vt = f["U" + side], f["Vt" + side]
            assert np.max(np.abs(U.T @ U - np.eye(s.rank))) < 1e-6
            assert np.max(np.abs(Vt @ Vt.T - np.eye(s.rank))) < 1e-6
            assert np.all(np.diff(f["s" + side]) <= 0)


@pytest.mark.parametrize("name", ["tiny-f32", "llama3-8b-layer-32k"])
def test_planted_needles_are_selected(name):
    case = make_case(WORKLOADS[name], variant="N")
    res = oracle.decode_step(**oracle_kwargs(case))
    for b in range(case.spec.batch):
        for g in range(case.spec.n_kv_heads):
            needles = set(case.needles[b, g][case.needles[b, g] >= 0].tolist())
            assert needles <= set(res["sel"][b, g].tolist())
    if case.spec.factor_kind == "gaussian":
        # planted outputs are O(1), literal ones tiny (the reason the planted variant exists)
        assert np.abs(res["out"]).max() > 0.1


def test_literal_layer_is_near_uniform():
    case = make_case(WORKLOADS["llama3-8b-layer-32k"])
    qd = from_storage(case.q, "bf16")
    kd = from_storage(case.sum_k[0, 0, :5], "bf16")
    assert np.abs(qd[0, 0] @ kd.T * case.spec.softmax_scale).max() < 1e-3
    assert math.isclose(case.spec.softmax_scale, 1 / math.sqrt(128))


def test_gate_inputs_are_deterministic_and_normalised():
    from synth import make_gate
    from synth.cases import from_storage
    case = make_case(custom_spec(dtype="f32", n_q_heads=4, n_kv_heads=2, head_dim=16, context=300, seed=41))
    a = make_gate(case, route_dim=8, tau="spread")
    b = make_gate(case, route_dim=8, tau="spread")
    assert np.array_equal(a.proj, b.proj) and np.array_equal(a.sum_route, b.sum_route)
    assert np.array_equal(a.thresholds, b.thresholds)
    kr = from_storage(a.sum_route, "f32")
    m = int(case.n_spans[0])
    assert np.allclose(np.linalg.norm(kr[0, :, :m], axis=-1), 1.0, atol=1e-6)
    assert np.all(kr[0, :, m:] == 0)
    p = make_gate(case, route_dim=8)
    assert np.all(p.tau == 0.05) and np.allclose(p.thresholds, np.log(0.05 / 0.95))


def test_adaptive_rank_arena_layout():
    from synth.cases import block_bytes, rank_granule
    for dt in ("f32", "bf16"):
        case = make_case(custom_spec(dtype=dt, n_q_heads=4, n_kv_heads=2, head_dim=32, rank=16, context=900,
                                     span_min=8, span_max=60, seed=44, rank_mode="adaptive"))
        gr = rank_granule(dt)
        ends = []
        for b in range(case.spec.batch):
            for g in range(case.spec.n_kv_heads):
                for S in range(int(case.n_spans[b])):
                    w = int(case.block_rank[b, g, S])
                    rk, rv = w & 0xFFFF, w >> 16
                    assert rk % gr == 0 and rv % gr == 0 and gr <= rk <= 16 and gr <= rv <= 16
                    o = int(case.block_off[b, g, S])
                    assert o % 256 == 0
                    ends.append((o, o + block_bytes(int(case.span_len[b, S]), rk, 32, dt, rv)))
        ends.sort()
        assert all(a[1] <= b[0] for a, b in zip(ends, ends[1:]))
        assert ends[-1][1] <= case.factors.nbytes
        fixed = make_case(custom_spec(dtype=dt, n_q_heads=4, n_kv_heads=2, head_dim=32, rank=16, context=900,
                                      span_min=8, span_max=60, seed=44))
        assert fixed.block_rank is None and case.factors.nbytes < fixed.factors.nbytes
