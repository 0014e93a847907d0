"""Seeded synthetic workloads for the split-head vocabulary projection.

This package only draws inputs (hidden states, LM-head weights, vocabulary
subsets, drafted tokens).  It holds none of the method's arithmetic: no
projection, clipping, quantisation, fusion, selection or verification.  Both
the CPU oracle's tests and the GPU path's tests and benchmark read their
inputs from here.
"""

from .workloads import (  # noqa: F401
    CONFIGS,
    Config,
    Workload,
    f32_to_bf16_bits,
    bf16_bits_to_f32,
    fp8_encode_rows,
    make_workload,
    with_subset,
    make_drafts,
    plant_masked_supertoken,
    scale_rows_bf16,
)
