"""CPU oracle for the split-head vocabulary projection.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow fp64 NumPy
restatement of the paper's distributed vocabulary projection (Section 5.4,
eqs. 9-15) and of the verification of drafted tokens (Section 5.5,
Algorithm 1).  It exists to check the HIP library; the library never calls
it.  Only the test suite, the package smoke check and the benchmark's CPU
baseline leg may import it.  It shares no code, table or constant generator
with the HIP path.

Parity status of each function (what pins it is listed in its docstring):
every function here is pinned by a CPU test under ``tests/``; the Philox
bit stream is pinned by published known-answer vectors of Philox4x32-10.
"""

from .split_head import (  # noqa: F401
    decode_bf16,
    decode_e4m3,
    full_head_logits,
    cloud_partial_logits,
    clip_quantize,
    clip_quantize_fmt,
    pack_codes,
    unpack_codes,
    payload_bytes,
    endpoint_partial_logits,
    hidden_quantize,
    endpoint_partial_logits_hq,
    fuse_masked,
    fuse_masked_fmt,
    round_sum_to_f32,
    greedy_select,
    philox4x32_10,
    philox_uniform,
    sample_select,
    sample_candidates,
    accept_lengths,
    cloud_call,
    endpoint_call,
)

from . import gcm  # noqa: F401,E402  (AES-GCM of eq. 19)
