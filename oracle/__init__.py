"""CPU oracle for LongNet dilated attention (forward and backward) and, in
layer_ref, the LongNet attention layer around it.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product path (the HIP library and its Python binding) never
calls it and shares no code with it.

Everything here is plain NumPy in float64, written to be checked against the
paper by eye rather than to be fast.
"""
from .dilated_ref import (  # noqa: F401
    head_offset,
    num_segments,
    segment_bounds,
    index_set,
    attend,
    per_pattern_ref,
    combine_ref,
    dilated_attention_ref,
    dilated_attention_rows_ref,
    default_scale,
)
from .brute import brute_mask_ref, brute_multiset_ref, visible_multiset  # noqa: F401
from .accounting import exact_causal_pairs, sparse_flops, covered_rows  # noqa: F401
from .dilated_bwd import (  # noqa: F401
    delta_ref,
    attend_bwd,
    dilated_attention_bwd_ref,
    dq_rows_ref,
    dkdv_rows_ref,
)
