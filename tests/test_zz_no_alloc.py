"""The allocation-free cloud call (sph_cloud_partial_noalloc) against the
call it varies (sph_cloud_partial_fmt with a caller workspace): both run the
same kernels, so payloads and partials must be identical bit for bit.  Two
calls in a row share the static scratch, the second with a smaller input;
a request larger than the scratch is refused before anything is launched."""

import sys

import numpy as np
import pytest
import torch

import paper_2607_13093_amd as sph
from paper_2607_13093_amd import _lib
from synth import Config, make_workload

import parity as P

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _both(dw, rows, bits, block):
    cfg = dw.cfg
    de = cfg.d_end
    h = dw.h[:rows]
    n = dw.subset.n
    nb = sph.payload_scale_count(n, block)
    q_ref, s_ref, z_ref = sph.cloud_partial(h[:, de:], dw.w_cloud, dw.subset, cfg.clip_c,
                                            w_row_scale=dw.w_scale, want_z=True, bits=bits,
                                            block=block)
    q = torch.empty_like(q_ref)
    s = torch.empty_like(s_ref)
    z = torch.empty_like(z_ref)
    sph.cloud_partial_noalloc(h[:, de:], dw.w_cloud, dw.subset, cfg.clip_c, out=(q, s, z),
                              w_row_scale=dw.w_scale, bits=bits, block=block)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(q), P.host(q_ref))
    np.testing.assert_array_equal(P.host(s).view(np.uint32), P.host(s_ref).view(np.uint32))
    np.testing.assert_array_equal(P.host(z).view(np.uint32), P.host(z_ref).view(np.uint32))
    assert nb == (1 if block == 0 else P.host(s).shape[1])


@pytest.mark.parametrize("wtype", ["bf16", "fp8"])
def test_noalloc_matches_the_workspace_call_twice(wtype):
    cfg = Config("noalloc", 91, d=1088, d_end=64, vocab=9000, n_sub=6001, subset_kind="choice",
                 sessions=40, rows_per_session=5, wtype=wtype)
    dw = P.DeviceWorkload(make_workload(cfg))
    # first call: 200 rows on the MFMA path; second call, smaller: 7 rows on
    # the skinny path; third: 40 rows, 4-bit codes with 256-position blocks
    for rows, bits, block in [(200, 8, 0), (7, 8, 0), (40, 4, 256)]:
        say(f"[gpu] noalloc {wtype}: {rows} rows, b={bits} block={block}")
        _both(dw, rows, bits, block)


def test_noalloc_refuses_more_than_its_scratch():
    cfg = Config("noalloc_big", 92, d=264, d_end=8, vocab=100000, n_sub=100000,
                 subset_kind="full", sessions=8, rows_per_session=6)
    dw = P.DeviceWorkload(make_workload(cfg))
    M = cfg.M  # 48 rows x 100000 ids: 19.2 MB of partials, more than the scratch
    assert sph.cloud_partial_workspace(M, dw.subset) > sph.api.NOALLOC_SCRATCH_BYTES
    q = torch.full((M, dw.subset.n), 7, dtype=torch.int8, device=dw.h.device)
    s = torch.full((M,), 3.0, dtype=torch.float32, device=dw.h.device)
    say("[gpu] noalloc: request beyond the scratch")
    with pytest.raises(sph.SphError) as ei:
        sph.cloud_partial_noalloc(dw.h[:, cfg.d_end:], dw.w_cloud, dw.subset, cfg.clip_c,
                                  out=(q, s, None))
    assert "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert int((q != 7).sum()) == 0 and float(s.max()) == 3.0   # nothing ran
    # a request that fits still runs after the refusal
    _both(dw, 5, 8, 0)
