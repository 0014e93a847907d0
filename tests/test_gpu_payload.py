"""GPU parity of the payload formats (b-bit codes, per-row or per-block
scales; eq. 18 and eq. 21) against the CPU oracle.

Each case runs both halves through the C ABI in one format and checks the
stages of tests/parity.py: A (partials), B (the oracle's quantiser and
packer applied to the GPU partials give the GPU payload byte for byte and
its scales bit for bit), C (codes vs the whole oracle's codes), D (the
oracle's dequantise + fuse + select of the GPU payload), E (whole pipelines).
Shapes cover the skinny projection (one and two row groups), the MFMA
projection with 128-, 256- and 320-row tiles, odd subset sizes (a 4-bit row
ending in a padding nibble), ragged last blocks and 16-byte-aligned payload
rows.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, Config, make_drafts, make_workload

import parity as P

pytestmark = pytest.mark.gpu

FORMATS = [(4, 0), (4, 256), (8, 256), (4, 1024), (8, 4096)]

SHAPES = [
    # (sessions, R, d, d_end, V, n)
    (1, 5, 1032, 8, 4000, 2501),     # skinny, odd n, ragged last block
    (13, 1, 1096, 72, 9000, 4097),   # skinny, two row groups, a last block of one position
    (3, 3, 520, 40, 3000, 1001),     # 9 rows: MFMA, 128-row tile
    (8, 5, 1032, 0, 4000, 2560),     # 40 rows, d_end = 0, 16-byte payload rows at b = 4
    (13, 10, 2056, 8, 9000, 8193),   # 130 rows: 256-row tile
    (24, 25, 1096, 72, 9000, 4097),  # 600 rows: two 320-row tiles, the second ragged
    # K a multiple of 64: at block 256 the projection's epilogue quantises
    (3, 3, 1088, 64, 5000, 2501),    # 9 rows: 32-row tile
    (8, 5, 1088, 64, 4000, 2560),    # 40 rows: 128-row tile
]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_format_case(wl, bits, block, tag, sessions=None):
    cfg = wl.cfg
    R = cfg.rows_per_session
    sess = np.arange(cfg.sessions) if sessions is None else np.asarray(sessions)
    rows = (sess[:, None] * R + np.arange(R)[None, :]).ravel()
    h_chk = wl.h_bits[rows]
    n = len(wl.subset)

    # whole oracle pipeline in this format
    orc = oracle.cloud_call(h_chk, cfg.d_end, wl.subset, cfg.clip_c, w_cloud_bits=wl.w_cloud_bits,
                            w_cloud_codes=wl.w_cloud_codes, w_cloud_scale=wl.w_cloud_scale,
                            bias=wl.bias, with_abs=True)
    orc_fmt = oracle.clip_quantize_fmt(orc["z"], cfg.clip_c, bits, block)
    z_e = oracle.endpoint_partial_logits(h_chk, cfg.d_end, wl.subset, wl.w_end_bits)[0]
    f_orc = oracle.fuse_masked_fmt(orc_fmt["q"], orc_fmt["scale"], z_e, block)
    ref_tok = np.zeros(cfg.M, np.int32)
    ref_tok[rows] = oracle.greedy_select(f_orc, wl.subset)[0]
    drafts_all = make_drafts(cfg, ref_tok, wl.subset) if cfg.k else None
    drafts = drafts_all[sess] if cfg.k else None

    say(f"[gpu] {tag}: cloud_partial bits={bits} block={block} M={cfg.M} d={cfg.d} "
        f"d_end={cfg.d_end} n={n}")
    dw = P.DeviceWorkload(wl)
    q, s, z = dw.cloud(bits=bits, block=block)
    torch.cuda.synchronize()
    nb = 1 if block == 0 else -(-n // block)
    assert tuple(q.shape) == (cfg.M, -(-n * bits // 8))
    assert tuple(s.shape) == ((cfg.M,) if block == 0 else (cfg.M, nb))
    qh, sh, zh = P.host(q)[rows], P.host(s)[rows], P.host(z)[rows]
    stats = {"A": P.stage_a(zh, orc)}
    codes = P.stage_b_fmt(zh, qh.view(np.uint8), sh, cfg.clip_c, bits, block)
    stats["C"] = P.stage_c_fmt(codes, sh, orc_fmt, orc["absdot"], block)

    say(f"[gpu] {tag}: fuse_verify bits={bits} block={block} sessions={cfg.sessions} R={R}")
    tok, acc, f = dw.fuse(q, s, drafts_all, bits=bits, block=block)
    torch.cuda.synchronize()
    th, ah, fh = P.host(tok)[rows], P.host(acc)[sess], P.host(f)[rows]
    wl2 = _with(wl, h_bits=h_chk, cfg=cfg.replace(sessions=len(sess)))
    s2 = sh.reshape(len(rows), nb)
    stats["D"] = P.stage_d_greedy(codes, s2, fh, th, ah, wl2, drafts, block=block)
    orc_e = {"q": orc_fmt["q"], "scale": orc_fmt["scale"]}
    stats["E"] = P.stage_e_greedy(codes, s2, th, ah, orc_e, wl2, drafts, block=block)
    say(f"[gpu] {tag}: ok {stats}")
    return stats


def _with(wl, **kw):
    import copy
    w2 = copy.copy(wl)
    for k, v in kw.items():
        setattr(w2, k, v)
    return w2


@pytest.mark.parametrize("fmt", FORMATS, ids=[f"b{b}blk{k}" for b, k in FORMATS])
@pytest.mark.parametrize("shape", SHAPES, ids=[f"S{s}R{r}d{d}de{de}V{v}n{n}" for s, r, d, de, v, n in SHAPES])
def test_payload_format_shapes(shape, fmt):
    S, R, d, de, V, n = shape
    bits, block = fmt
    cfg = Config("payload", 60 + sum(shape) + bits + block % 97, d=d, d_end=de, vocab=V, n_sub=n,
                 subset_kind="choice", sessions=S, rows_per_session=R)
    run_format_case(make_workload(cfg), bits, block, f"payload {shape} b={bits} block={block}")


def test_payload_format_fp8_weights():
    cfg = Config("payload_fp8", 71, d=1088, d_end=64, vocab=7000, n_sub=3003, subset_kind="choice",
                 sessions=60, rows_per_session=5, wtype="fp8", with_bias=True)
    run_format_case(make_workload(cfg), 4, 256, "payload fp8 300 rows b=4 block=256")


@pytest.mark.parametrize("name", ["decode", "dense_sub"])
def test_payload_format_benchmark_workloads(name):
    # the benchmark launches in the 4-bit, 256-position-block format; the
    # dense one is checked on four whole sessions
    wl = make_workload(CONFIGS[name])
    sessions = None if name == "decode" else [0, 77, 160, 255]
    run_format_case(wl, 4, 256, f"{name} b=4 block=256", sessions=sessions)


def test_payload_format_sampling():
    # the sampler consumes fused logits of a 4-bit payload with block scales
    cfg = Config("payload_sample", 73, d=520, d_end=40, vocab=9000, n_sub=8191,
                 subset_kind="choice", sessions=5, rows_per_session=3, mode="sample",
                 temperature=0.7, top_p=0.9, philox_seed=0x0DDC0FFEE)
    wl = make_workload(cfg)
    bits, block = 4, 256
    rows = np.arange(cfg.M)
    orc = oracle.cloud_call(wl.h_bits, cfg.d_end, wl.subset, cfg.clip_c,
                            w_cloud_bits=wl.w_cloud_bits, with_abs=True)
    z_e, absdot_e = oracle.endpoint_partial_logits(wl.h_bits, cfg.d_end, wl.subset, wl.w_end_bits,
                                                   with_abs=True)
    drafts = np.zeros((cfg.sessions, cfg.k), np.int32)
    say(f"[gpu] payload sampling: M={cfg.M} n={len(wl.subset)} b={bits} block={block}")
    dw = P.DeviceWorkload(wl)
    q, s, z = dw.cloud(bits=bits, block=block)
    tok, acc, f = dw.fuse(q, s, drafts, bits=bits, block=block)
    torch.cuda.synchronize()
    zh, qh, sh = P.host(z), P.host(q), P.host(s)
    th, ah, fh = P.host(tok), P.host(acc), P.host(f)
    P.stage_a(zh, orc)
    codes = P.stage_b_fmt(zh, qh.view(np.uint8), sh, cfg.clip_c, bits, block)
    f_ref = oracle.fuse_masked_fmt(codes, sh, z_e, block)
    df = np.abs(fh.astype(np.float64) - f_ref.astype(np.float64))
    assert (df <= P.tol_of(absdot_e) + P.ULP * np.abs(f_ref)).all(), "fused logits"
    tok_ref, info = oracle.sample_select(fh, wl.subset, cfg.temperature, cfg.top_p,
                                         cfg.philox_seed, cfg.rows_per_session, row_index=rows)
    exempt = (info["cut_margin"] <= 1e-9) | (info["cdf_margin"] <= 1e-9)
    bad = (th != tok_ref) & ~exempt
    assert not bad.any(), f"{bad.sum()} sampled tokens differ"
    P.check_boundary_rows(th, tok_ref, fh, wl.subset, cfg, rows, 1e-9)
    np.testing.assert_array_equal(ah, oracle.accept_lengths(th, drafts, cfg.sessions,
                                                            cfg.rows_per_session))
    say(f"[gpu] payload sampling: ok, exempt {int(exempt.sum())}")


@pytest.mark.parametrize("bits", [8, 4])
def test_epilogue_quantiser_without_z(bits):
    # block 256 on the MFMA path: the payload is the same whether or not the
    # fp32 partials are also written
    cfg = Config("payload_noz", 74, d=2112, d_end=64, vocab=9000, n_sub=6001, subset_kind="choice",
                 sessions=60, rows_per_session=5)
    wl = make_workload(cfg)
    dw = P.DeviceWorkload(wl)
    say(f"[gpu] epilogue quantiser b={bits}: with and without z")
    q1, s1, z1 = dw.cloud(want_z=True, bits=bits, block=256)
    q2, s2, z2 = dw.cloud(want_z=False, bits=bits, block=256)
    torch.cuda.synchronize()
    assert z2 is None
    np.testing.assert_array_equal(P.host(q1), P.host(q2))
    np.testing.assert_array_equal(P.host(s1).view(np.uint32), P.host(s2).view(np.uint32))
    codes = P.stage_b_fmt(P.host(z1), P.host(q1).view(np.uint8), P.host(s1), cfg.clip_c, bits, 256)
    assert codes.shape == (cfg.M, len(wl.subset))
