"""Split-head vocabulary projection (distributed LM head with speculative
verification) as hand-written HIP kernels for MI355X / gfx950.

The library is libsph.so (C ABI, include/sph.h); this package is its thin
torch binding.  Importing it does not touch the GPU.
"""

from .api import (  # noqa: F401
    GREEDY,
    SAMPLE,
    SphError,
    Subset,
    cloud_partial,
    cloud_partial_workspace,
    cloud_partial_noalloc,
    debug_sync,
    fuse_verify,
    fuse_verify_workspace,
    payload_code_bytes,
    hidden_quantize,
    GcmKey,
    gcm_seal,
    gcm_open,
    gcm_seal_segments,
    gcm_open_segments,
    gcm_workspace,
    fuse_verify_hq,
    fuse_verify_hq_workspace,
    payload_scale_count,
    probe_mfma,
    probe_read,
    trace_collect,
    trace_start,
)
