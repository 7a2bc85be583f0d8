"""fp64 CPU oracle for block selection and block-sparse attention.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the package smoke check and the
bench's CPU-baseline leg may import this package.  The GPU library never calls
it, and it shares no code with the GPU library.
"""
from .la_oracle import (  # noqa: F401
    bf16_bits_to_f64,
    partition,
    pool_blocks,
    block_scores,
    softmax_rows,
    select_tau_row,
    select_topk_row,
    select_blocks,
    ambiguous_blocks,
    visible_keys,
    attention_block,
    attention,
    attention_rows,
    kept_flops,
)
