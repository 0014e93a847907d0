"""The two calls captured in a HIP graph (torch.cuda.graph) and replayed,
also with the payload sealed and opened between them.

Every call only enqueues kernels on the caller's stream (no allocation,
memset or synchronisation inside), so the whole step can be captured.  Each
replay is compared bit for bit with the eager results, with eager work of
the program between the replays; the captured step runs on pre-allocated
outputs and workspaces."""

import sys

import numpy as np
import pytest
import torch

import paper_2607_13093_amd as sph
from synth import CONFIGS, Config, make_drafts, make_workload

import parity as P

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _step_buffers(dw, cfg, sub, M, n, bits, block):
    dev = torch.device("cuda")
    nb = sph.payload_scale_count(n, block)
    q = torch.empty((M, sph.payload_code_bytes(n, bits)), dtype=torch.uint8, device=dev)
    s = torch.empty((M,) if block == 0 else (M, nb), dtype=torch.float32, device=dev)
    tok = torch.empty((M,), dtype=torch.int32, device=dev)
    acc = torch.empty((cfg.sessions,), dtype=torch.int32, device=dev)
    f = torch.empty((M, n), dtype=torch.float32, device=dev)
    ws_c = torch.empty(max(1, sph.cloud_partial_workspace(M, sub)), dtype=torch.uint8, device=dev)
    ws_f = torch.empty(max(1, sph.fuse_verify_workspace(M, sub, sph.GREEDY)), dtype=torch.uint8, device=dev)
    return q, s, tok, acc, f, ws_c, ws_f


@pytest.mark.parametrize("name,bits,block,sealed", [("decode", 8, 0, False), ("batched_small", 4, 256, False),
                                                     ("decode_sealed", 8, 0, True)])
def test_step_in_a_graph_replays_exactly(name, bits, block, sealed):
    if name.startswith("decode"):
        cfg = CONFIGS["decode"]
    else:   # 40 rows: the MFMA path in both calls
        cfg = Config("graph", 97, d=1032, d_end=64, vocab=6000, n_sub=2560, subset_kind="choice",
                     sessions=8, rows_per_session=5)
    wl = make_workload(cfg)
    dw = P.DeviceWorkload(wl)
    M, n, de = cfg.M, len(wl.subset), cfg.d_end
    drafts = P.to_dev(make_drafts(cfg, np.zeros(M, np.int32), wl.subset))
    q, s, tok, acc, f, ws_c, ws_f = _step_buffers(dw, cfg, dw.subset, M, n, bits, block)
    outs = [q, s, tok, acc, f]
    if sealed:
        # the payload crosses as one AES-GCM message per row (codes, then
        # scales) and the endpoint works on the opened copy
        key = sph.GcmKey(bytes(range(32)))
        s_b = s.view(torch.uint8).reshape(M, -1)
        cq, cs = torch.empty_like(q), torch.empty_like(s_b)
        q2, s2 = torch.empty_like(q), torch.empty_like(s)
        s2_b = s2.view(torch.uint8).reshape(M, -1)
        tag = torch.empty((M, 16), dtype=torch.uint8, device="cuda")
        ok = torch.empty((M,), dtype=torch.int32, device="cuda")
        iv = P.to_dev(np.arange(M * 12, dtype=np.uint32).astype(np.uint8).reshape(M, 12))
        aad = P.to_dev(np.full((M, 20), 7, np.uint8))
        ws_g = torch.empty(max(1, sph.gcm_workspace(M, q.shape[1] + s_b.shape[1])), dtype=torch.uint8,
                           device="cuda")
        outs += [cq, cs, tag, ok, q2, s2]

    def step():
        sph.cloud_partial(dw.h[:, de:], dw.w_cloud, dw.subset, cfg.clip_c, workspace=ws_c,
                          out=(q, s, None), bits=bits, block=block)
        qe, se = q, s
        if sealed:
            sph.gcm_seal_segments(key, (q, s_b), iv, aad, out=(cq, cs), tag=tag, workspace=ws_g)
            sph.gcm_open_segments(key, (cq, cs), iv, tag, aad, out=(q2, s2_b), ok=ok, workspace=ws_g)
            qe, se = q2, s2
        sph.fuse_verify(qe, se, dw.h[:, :de], dw.w_end, dw.subset, cfg.sessions, cfg.rows_per_session,
                        drafts, workspace=ws_f, out=(tok, acc, f), want_fused=True, bits=bits, block=block)

    say(f"[gpu] graph {name}: eager")
    step()
    torch.cuda.synchronize()
    ref = [P.host(t).copy() for t in outs]
    if sealed:                                  # outs: q s tok acc f cq cs tag ok q2 s2
        assert ref[8].tolist() == [1] * M
        np.testing.assert_array_equal(ref[9], ref[0])
        np.testing.assert_array_equal(ref[10].view(np.uint8), ref[1].view(np.uint8))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                                  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say(f"[gpu] graph {name}: capture")
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in outs:                           # program work between replays
            t.zero_()
        torch.cuda.synchronize()
        say(f"[gpu] graph {name}: replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        for r, t in zip(ref, outs):
            np.testing.assert_array_equal(P.host(t).view(np.uint8), r.view(np.uint8))
    g.reset()
