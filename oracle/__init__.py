"""CPU oracle of the SeKV decode step.  Test infrastructure only: imported by
the tests, the smoke check and the benchmark's CPU-baseline leg, never by the
product path."""

from .sekv_oracle import (  # noqa: F401
    block_ranks,
    decode_step,
    deploy_factors,
    decode_step_gated,
    gate,
    gate_logits,
    gated_reconstruct,
    gated_selection,
    group_keys,
    merge_partials,
    mixed_attention_head,
    project_queries,
    read_span_block,
    reconstruct,
    routing_logits,
    select_topk,
    softmax_partial,
    softmax_weights,
    summary_key,
    surprisal_weights,
    threshold_logit,
    widen,
    zoom_attend,
    zoom_scores_factored,
    zoom_values_factored,
)
