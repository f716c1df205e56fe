"""CPU oracle of the SeKV decode step.  Test infrastructure only: imported by
the tests, the smoke check and the benchmark's CPU-baseline leg, never by the
product path."""

from .sekv_oracle import (  # noqa: F401
    decode_step,
    group_keys,
    merge_partials,
    mixed_attention_head,
    read_span_block,
    reconstruct,
    routing_logits,
    select_topk,
    softmax_partial,
    softmax_weights,
    widen,
    zoom_attend,
    zoom_scores_factored,
    zoom_values_factored,
)
