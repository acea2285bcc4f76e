"""CPU oracle for Sparse Reference Attention — test infrastructure only.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
package; the product path never does.
"""
from .sra_oracle import (  # noqa: F401
    attention_backward_full,
    attention_rows,
    default_scale,
    dkv_keys,
    dq_rows,
    forward_rows,
    frame_valid,
    pair_counts,
    sample_sizes,
    sra_backward,
    sra_forward,
    visibility_mask,
)
