"""Seeded synthetic SeKV caches.

This package builds the stored inputs of one decode step (query, anchor K/V,
span summaries, span factor blocks and the span tables) for the workload
shapes the decode-step tests and benchmark use.  It plays the part of the
paper's prefill stage for synthetic data only: it draws values, partitions the
context into spans, and forms each span's coarse mean key/value and, for the
learned selection rule, random routing projections, the projected normalised
routing summaries and the zoom thresholds; and, for the prefill-side builder,
token keys/values and surprisal.  It holds
none of the decode step's arithmetic (routing, selection, reconstruction for
attention, softmax), and it imports neither the oracle nor the HIP library.
"""

from .cases import (  # noqa: F401
    WORKLOADS,
    case_from_factors,
    with_top_k,
    Case,
    CaseSpec,
    bf16_bits_to_f64,
    custom_spec,
    f64_to_bf16_bits,
    make_case,
    Gate,
    NO_BUDGET,
    make_gate,
    Prefill,
    make_prefill,
)
