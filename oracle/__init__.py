"""CPU oracle of the joint-evaluation forward pass (float64, numpy).

TEST INFRASTRUCTURE ONLY: imported by tests, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.
"""
from .evaluator import (  # noqa: F401
    LN_EPS, layer_norm, softmax_rows, attention, elu_plus_one, linear_attention, linear_kv_state, attend,
    module_attention, self_attention_block, ffn, encoder_block,
    encoder_stack, context_rows, encode_context, distinct_items, item_rows, encode_items,
    assemble_one, encode_sequence, cross_sequence, score, score_objectives, select, evaluate_naive,
    evaluate_cached,
)
from .brute import evaluate_brute  # noqa: F401
