"""Determinism of the HIP path across launch geometries, and the debug
synchronisation mode.

The same verification session (5 rows) is placed, at different row offsets,
into batches of 5, 20, 100, 300 and 400 rows, which the library runs with
the skinny VALU kernel and with 32-, 128-, 320- and 256-row MFMA tiles (the
last one with the session straddling two row tiles).  Every MFMA tile adds
the products of an output element in the same order (K steps of 64, the
32x32x16 instruction's 16 products per step), so the session's fp32
partials, payload, fused logits, tokens and accept length must be bit
identical across the four MFMA geometries.  The skinny kernel sums in
another order: its partials agree within the fp32 tolerance and its tokens
equal the MFMA ones unless a competitor lies within that bound.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_13093_amd as sph
from synth import Config, make_drafts, make_workload

import parity as P

pytestmark = pytest.mark.gpu

R = 5
# (batch rows, row offset of the session): skinny, then MFMA tiles of 32,
# 128, 320 and 256 rows (255..259 straddles the first 256-row boundary)
GEOMETRIES = [(5, 0), (20, 15), (100, 60), (300, 250), (400, 255)]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _case():
    cfg = Config("geom", 81, d=1088, d_end=64, vocab=6000, n_sub=4001, subset_kind="choice",
                 sessions=80, rows_per_session=R)
    wl = make_workload(cfg)              # 400 rows of h; rows 0..4 are the session
    return cfg, wl


def _run(cfg, wl, dw, M, off, drafts_one):
    # batch: filler rows from the workload's pool, the session at `off`
    idx = np.arange(R, R + M) % cfg.M
    idx[off:off + R] = np.arange(R)
    h = dw.h[torch.from_numpy(idx).to(dw.h.device)]
    de = cfg.d_end
    q, s, z = sph.cloud_partial(h[:, de:], dw.w_cloud, dw.subset, cfg.clip_c, want_z=True)
    S = M // R
    drafts = torch.zeros((S, R - 1), dtype=torch.int32, device=dw.h.device)
    drafts[off // R] = torch.from_numpy(drafts_one).to(dw.h.device)
    tok, acc, f = sph.fuse_verify(q, s, h[:, :de], dw.w_end, dw.subset, S, R, drafts,
                                  want_fused=True)
    torch.cuda.synchronize()
    sl = slice(off, off + R)
    return {"z": P.host(z)[sl], "q": P.host(q)[sl], "s": P.host(s)[sl], "f": P.host(f)[sl],
            "tok": P.host(tok)[sl], "acc": int(P.host(acc)[off // R])}


def test_results_across_launch_geometries():
    cfg, wl = _case()
    dw = P.DeviceWorkload(wl)
    orc = oracle.cloud_call(wl.h_bits[:R], cfg.d_end, wl.subset, cfg.clip_c,
                            w_cloud_bits=wl.w_cloud_bits, with_abs=True)
    ep = oracle.endpoint_call(orc["q"], orc["scale"], wl.h_bits[:R], cfg.d_end, wl.subset,
                              wl.w_end_bits, 1, R, drafts=np.zeros((1, R - 1), np.int32))
    one = cfg.replace(sessions=1)
    drafts_one = make_drafts(one, ep["tokens"], wl.subset)[0]
    res = {}
    for M, off in GEOMETRIES:
        say(f"[gpu] geometry M={M} session rows {off}..{off + R - 1}")
        res[M] = _run(cfg, wl, dw, M, off, drafts_one)
    ref = res[20]
    for M in (100, 300, 400):
        r = res[M]
        for k in ("z", "f"):
            np.testing.assert_array_equal(r[k].view(np.uint32), ref[k].view(np.uint32),
                                          err_msg=f"{k} differs between MFMA tiles (M={M})")
        np.testing.assert_array_equal(r["q"], ref["q"])
        np.testing.assert_array_equal(r["s"].view(np.uint32), ref["s"].view(np.uint32))
        np.testing.assert_array_equal(r["tok"], ref["tok"])
        assert r["acc"] == ref["acc"]
    # every geometry against the oracle (stage A), and the skinny run's
    # tokens against the MFMA ones where no competitor is within the bound
    for M, r in res.items():
        P.stage_a(r["z"], orc)
        P.stage_b(r["z"], r["q"], r["s"], cfg.clip_c)
    sk = res[5]
    z_e, absdot = oracle.endpoint_partial_logits(wl.h_bits[:R], cfg.d_end, wl.subset,
                                                 wl.w_end_bits, with_abs=True)
    f_ref = oracle.fuse_masked(ref["q"], ref["s"], z_e)
    bound = P.tol_of(absdot) + P.ULP * np.abs(f_ref.astype(np.float64))
    ex = P.exempt_rows(f_ref, bound)
    if not (sk["q"] != ref["q"]).any():
        assert not ((sk["tok"] != ref["tok"]) & ~ex).any(), "skinny and MFMA tokens differ"
    say(f"[gpu] geometries ok: exempt rows {int(ex.sum())}, "
        f"skinny code differences {int((sk['q'] != ref['q']).sum())}")


def test_debug_sync_gives_the_same_results():
    cfg, wl = _case()
    dw = P.DeviceWorkload(wl)
    drafts_one = np.zeros(R - 1, np.int32)
    say("[gpu] debug sync off / on, M=5 and M=100")
    prev = sph.debug_sync(False)
    try:
        off = {M: _run(cfg, wl, dw, M, o, drafts_one) for M, o in [(5, 0), (100, 60)]}
        assert sph.debug_sync(True) is False
        on = {M: _run(cfg, wl, dw, M, o, drafts_one) for M, o in [(5, 0), (100, 60)]}
    finally:
        sph.debug_sync(prev)
    for M in off:
        for k in ("z", "q", "s", "f", "tok"):
            np.testing.assert_array_equal(np.asarray(on[M][k]), np.asarray(off[M][k]))
        assert on[M]["acc"] == off[M]["acc"]
