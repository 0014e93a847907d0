"""GPU parity of libsph against the CPU oracle (staged: see tests/parity.py).

Every test here calls the HIP library through its C ABI; none has a CPU
fallback.  Case names are printed (and flushed) before each GPU step.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_13093_amd as sph
from paper_2607_13093_amd import _lib
from synth import (CONFIGS, Config, make_drafts, make_workload, plant_masked_supertoken,
                   scale_rows_bf16)

import parity as P

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_greedy_case(wl, h_bits=None, w_end_bits=None, w_cloud_bits=None, tag="", sessions=None,
                    dw=None):
    """Full staged parity A-E of one greedy workload; returns the stats.

    The GPU always runs the whole workload (the launch configuration of the
    benchmark); with `sessions` the oracle checks only those sessions' rows
    (rows are independent, and whole sessions keep accept lengths checkable).
    `dw`: the workload's device tensors, when the test lays them out itself.
    """
    cfg = wl.cfg
    h_bits = wl.h_bits if h_bits is None else h_bits
    w_end_bits = wl.w_end_bits if w_end_bits is None else w_end_bits
    w_cloud_bits = wl.w_cloud_bits if w_cloud_bits is None else w_cloud_bits
    R = cfg.rows_per_session
    sess = np.arange(cfg.sessions) if sessions is None else np.asarray(sessions)
    rows = (sess[:, None] * R + np.arange(R)[None, :]).ravel()
    h_chk = h_bits[rows]
    orc = oracle.cloud_call(h_chk, cfg.d_end, wl.subset, cfg.clip_c, w_cloud_bits=w_cloud_bits,
                            w_cloud_codes=wl.w_cloud_codes, w_cloud_scale=wl.w_cloud_scale,
                            bias=wl.bias, with_abs=True)
    ep = oracle.endpoint_call(orc["q"], orc["scale"], h_chk, cfg.d_end, wl.subset, w_end_bits,
                              len(sess), R, drafts=np.zeros((len(sess), cfg.k), np.int32))
    ref_tok = np.zeros(cfg.M, np.int32)
    ref_tok[rows] = ep["tokens"]
    drafts_all = make_drafts(cfg, ref_tok, wl.subset) if cfg.k else None
    drafts = drafts_all[sess] if cfg.k else None

    say(f"[gpu] {tag or cfg.name}: cloud_partial M={cfg.M} d={cfg.d} d_end={cfg.d_end} "
        f"n={len(wl.subset)} wtype={cfg.wtype}")
    if dw is None:
        dw = P.DeviceWorkload(wl, h_bits=h_bits, w_end_bits=w_end_bits, w_cloud_bits=w_cloud_bits)
    q, s, z = dw.cloud()
    torch.cuda.synchronize()
    qh, sh, zh = P.host(q)[rows], P.host(s)[rows], P.host(z)[rows]
    stats = {"A": P.stage_a(zh, orc)}
    P.stage_b(zh, qh, sh, cfg.clip_c)
    stats["C"] = P.stage_c(qh, sh, orc)

    say(f"[gpu] {tag or cfg.name}: fuse_verify sessions={cfg.sessions} R={R}")
    tok, acc, f = dw.fuse(q, s, drafts_all)
    torch.cuda.synchronize()
    th, ah, fh = P.host(tok)[rows], P.host(acc)[sess], P.host(f)[rows]
    wl2 = _with(wl, h_bits=h_chk, w_end_bits=w_end_bits, cfg=cfg.replace(sessions=len(sess)))
    stats["D"] = P.stage_d_greedy(qh, sh, fh, th, ah, wl2, drafts)
    stats["E"] = P.stage_e_greedy(qh, sh, th, ah, orc, wl2, drafts)
    say(f"[gpu] {tag or cfg.name}: ok {stats}")
    return stats, (qh, sh, zh, th, ah, fh)


def _with(wl, **kw):
    import copy
    w2 = copy.copy(wl)
    for k, v in kw.items():
        setattr(w2, k, v)
    return w2


# ---------------------------------------------------------------------------
# the benchmark workloads
# ---------------------------------------------------------------------------

def test_tiny_full_pipeline():
    run_greedy_case(make_workload(CONFIGS["tiny"]))


def test_decode_full_pipeline():
    run_greedy_case(make_workload(CONFIGS["decode"]))


def test_batched_full_pipeline():
    run_greedy_case(make_workload(CONFIGS["batched"]))


# One whole session in each 256-row tile of the 2048-row launch (session s
# holds rows 8s .. 8s+7, so sessions 0, 32, ..., 224 open tiles 0 .. 7),
# plus the last session.
DENSE_SESSIONS = list(range(0, 256, 32)) + [255]


@pytest.mark.parametrize("name", ["dense_full", "dense_sub"])
def test_dense_sampled_sessions(name):
    # the full 2048-row launch, as the benchmark runs it; the oracle checks
    # 9 whole sessions (72 rows) spread over every row tile
    run_greedy_case(make_workload(CONFIGS[name]), sessions=DENSE_SESSIONS)


@pytest.mark.parametrize("d_end", [48, 96])
def test_paper_shape_full_vocabulary(d_end):
    # the paper's evaluation shape (Section 7.3): hidden 4096, a vocabulary of
    # 150000 ids with every id kept (the mixed-language mode), d_end 48 or 96
    # (Table 6), one session verifying k = 4 drafts
    cfg = Config("paper_shape", 60 + d_end, d=4096, d_end=d_end, vocab=150000, n_sub=150000,
                 subset_kind="full", sessions=1, rows_per_session=5)
    run_greedy_case(make_workload(cfg), tag=f"paper shape d_end={d_end}")


@pytest.mark.parametrize("wtype", ["bf16", "fp8"])
def test_weights_beyond_4gib_of_their_base(wtype):
    # weight rows more than 4 GiB past the start of the weights: the
    # direct-to-LDS projections then address their copies with 64-bit lane
    # addresses instead of 32-bit offsets from a scalar base (40 rows: the
    # MFMA path in both calls; bf16 or E4M3 cloud weights)
    cfg = Config("wide", 71, d=1088, d_end=64, vocab=70000, n_sub=20000, subset_kind="choice",
                 sessions=8, rows_per_session=5, wtype=wtype)
    wl = make_workload(cfg)
    dw = P.DeviceWorkload(wl)
    row_bytes = 65536  # 70000 rows of 64 KiB: 4.6 GB
    dc, de = cfg.d - cfg.d_end, cfg.d_end
    wc = torch.empty((cfg.vocab, row_bytes // dw.w_cloud.element_size()), dtype=dw.w_cloud.dtype,
                     device="cuda")
    wc[:, :dc] = dw.w_cloud
    we = torch.empty((cfg.vocab, row_bytes // 2), dtype=torch.bfloat16, device="cuda")
    we[:, :de] = dw.w_end
    dw.w_cloud, dw.w_end = wc[:, :dc], we[:, :de]
    assert int(np.max(wl.subset)) * row_bytes > 2 ** 32
    run_greedy_case(wl, tag=f"{wtype} weights beyond 4 GiB", dw=dw)
    del wc, we, dw
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# shapes: ragged tails, row groups, d_end = 0, bias, k = 0
# ---------------------------------------------------------------------------

RAGGED = [
    # (sessions, R, d, d_end, V, n)
    (1, 1, 64, 8, 300, 1),
    (1, 2, 72, 16, 500, 7),
    (1, 7, 520, 40, 3000, 1001),
    (2, 4, 1032, 8, 4000, 2500),
    (3, 3, 264, 0, 2000, 777),      # d_end = 0: the cloud computes the whole head
    (13, 1, 136, 64, 1000, 333),    # 13 rows: two row groups
    (4, 5, 4104, 520, 6000, 4097),  # d_end > 512 and a ragged subset
    (3, 1, 8192, 512, 3000, 2999),  # four passes over each cloud row
    # dense (MFMA) path: more than 8 rows
    (3, 3, 520, 40, 3000, 1001),    # 9 rows, ragged m- and n-tiles
    (8, 5, 1032, 0, 4000, 2500),    # 40 rows, d_end = 0
    (17, 17, 1096, 72, 9000, 4097), # 289 rows: one 320-row m-tile (8 waves), ragged n
    (24, 25, 1096, 72, 9000, 4097), # 600 rows: two 320-row m-tiles, the second ragged
    (13, 10, 2056, 8, 9000, 8193),  # 130 rows: two m-tiles, last n-tile of one column
    # 256-row tiles at the edges of the one-wave kernel's step counts
    (32, 8, 128, 64, 3000, 1001),   # one K step (the two-wave kernel)
    (32, 8, 192, 64, 3000, 1001),   # two K steps (one wave, two weight stages)
    (32, 8, 448, 64, 3000, 1001),   # six K steps (one wave, three weight stages)
    # 32-row tiles (9..32 rows, K a multiple of 64 in both calls)
    (3, 3, 1088, 64, 5000, 2501),   # 9 rows
    (4, 8, 2304, 256, 9000, 4097),  # 32 rows, ragged n
    (1, 9, 4096, 256, 20000, 9001), # the decode step with k = 8 drafts
]


@pytest.mark.parametrize("shape", RAGGED, ids=[f"S{s}R{r}d{d}de{de}V{v}n{n}" for s, r, d, de, v, n in RAGGED])
def test_ragged_shapes(shape):
    S, R, d, de, V, n = shape
    cfg = Config("ragged", 10 + sum(shape), d=d, d_end=de, vocab=V, n_sub=n, subset_kind="choice",
                 sessions=S, rows_per_session=R)
    run_greedy_case(make_workload(cfg), tag=f"ragged {shape}")


def test_bias_is_added_once_on_the_cloud():
    cfg = CONFIGS["tiny"].replace(name="tiny_bias", with_bias=True)
    run_greedy_case(make_workload(cfg), tag="bias")


def test_full_vocabulary_plan():
    cfg = Config("full_small", 21, d=256, d_end=32, vocab=3000, n_sub=3000, subset_kind="full",
                 sessions=2, rows_per_session=4)
    run_greedy_case(make_workload(cfg), tag="full-vocab")


def test_clip_zero_and_masked_supertoken_rows():
    cfg = Config("edge", 22, d=512, d_end=64, vocab=8192, n_sub=4096, subset_kind="perm",
                 sessions=2, rows_per_session=3)
    wl = make_workload(cfg)
    h = scale_rows_bf16(wl.h_bits, [0, 4], 10.0)     # clipped rows
    h[2] = 0                                          # a zero row
    we, wc = wl.w_end_bits.copy(), wl.w_cloud_bits.copy()
    vid = plant_masked_supertoken(we, wc, h, 1, wl.subset)
    stats, (q, s, z, tok, acc, f) = run_greedy_case(wl, h_bits=h, w_end_bits=we, w_cloud_bits=wc,
                                                    tag="clip/zero/planted")
    assert s[0] == np.float32(30.0) / np.float32(127.0) and s[4] == s[0]
    assert s[2] == 0 and not q[2].any()
    assert tok[2] == wl.subset[0]          # an all-zero row ties everywhere: lowest id wins
    assert vid not in tok


# Tie rows on the MFMA endpoint path (128-, 320- and 256-row tiles): h row
# e_c makes the cloud partial 0 (so q = 0, s = 0) and the fused logit of
# position j equal to W_end[S_j, c] exactly; column c holds -1 except +1 at
# the positions of pattern c.  The patterns put the maxima 32 positions apart
# (one lane, two column slots of a tile), in two lanes of one tile, in two
# tiles (one of them the ragged last), and three apart.  All-zero rows tie
# at every position.  Eq. 15 with the lowest-id reading of ties.
TIE_PATTERNS = [(5, 37), (300, 290), (2999, 700), (40, 8, 2000)]


@pytest.mark.parametrize("rows,tie_rows,zero_row", [
    (48, (0, 7, 20, 47), 30),
    (300, (0, 130, 257, 299), 150),
    (512, (0, 255, 256, 511), 100),
], ids=["M48", "M300", "M512"])
def test_mfma_endpoint_ties_go_to_the_lowest_id(rows, tie_rows, zero_row):
    cfg = Config("ties_mfma", 40 + rows, d=256, d_end=64, vocab=6000, n_sub=3000,
                 subset_kind="choice", sessions=rows // 4, rows_per_session=4)
    wl = make_workload(cfg)
    one, minus_one = np.uint16(0x3F80), np.uint16(0xBF80)   # bf16 +1, -1
    h = wl.h_bits.copy()
    we = wl.w_end_bits.copy()
    for c, (r, pat) in enumerate(zip(tie_rows, TIE_PATTERNS)):
        h[r] = 0
        h[r, c] = one
        we[wl.subset, c] = minus_one
        we[wl.subset[list(pat)], c] = one
    h[zero_row] = 0
    stats, (q, s, z, tok, acc, f) = run_greedy_case(wl, h_bits=h, w_end_bits=we,
                                                    tag=f"endpoint ties M={rows}")
    for r, pat in zip(tie_rows, TIE_PATTERNS):
        assert s[r] == 0 and not q[r].any()
        assert tok[r] == wl.subset[min(pat)], (r, pat, tok[r])
    assert tok[zero_row] == wl.subset[0]


# ---------------------------------------------------------------------------
# fp8 cloud weights
# ---------------------------------------------------------------------------

def test_fp8_decode_of_every_code_through_the_abi():
    # W row v holds code v in column 0 and zeros elsewhere; h is the unit vector e_0,
    # so z[v] = decode(code_v) * 1.0 exactly.  NaN codes are left out.
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    V, K = codes.size, 16
    w = np.zeros((V, K), np.uint8)
    w[:, 0] = codes
    h = np.zeros((1, K), np.uint16)
    h[0, 0] = 0x3F80  # bf16 1.0
    say("[gpu] fp8 decode: all finite E4M3 codes")
    sub = sph.Subset(np.arange(V), vocab=V)
    q, s, z = sph.cloud_partial(P.to_dev(h, torch.bfloat16), P.to_dev(w, torch.uint8), sub, 1000.0,
                                w_row_scale=torch.ones(V, device="cuda"), want_z=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(z)[0], oracle.decode_e4m3(codes).astype(np.float32))


def test_fp8_cloud_partial_skinny():
    cfg = Config("fp8_small", 23, d=1056, d_end=32, vocab=5000, n_sub=2048, subset_kind="choice",
                 sessions=1, rows_per_session=5, wtype="fp8")
    run_greedy_case(make_workload(cfg), tag="fp8 skinny")


def test_fp8_cloud_partial_dense():
    cfg = Config("fp8_dense", 27, d=1056, d_end=32, vocab=5000, n_sub=3001, subset_kind="choice",
                 sessions=12, rows_per_session=5, wtype="fp8", with_bias=True)
    run_greedy_case(make_workload(cfg), tag="fp8 dense")


def test_fp8_cloud_partial_dense_320_row_tiles():
    # 300 rows: one 320-row tile of 8 waves, fp8 codes copied to LDS directly
    cfg = Config("fp8_dense_320", 29, d=1088, d_end=64, vocab=7000, n_sub=3003, subset_kind="choice",
                 sessions=60, rows_per_session=5, wtype="fp8", with_bias=True)
    run_greedy_case(make_workload(cfg), tag="fp8 dense, 320-row tiles")


def test_fp8_cloud_partial_32_row_tiles():
    cfg = Config("fp8_32", 31, d=1088, d_end=64, vocab=5000, n_sub=3001, subset_kind="choice",
                 sessions=4, rows_per_session=5, wtype="fp8", with_bias=True)
    run_greedy_case(make_workload(cfg), tag="fp8, 20 rows in a 32-row tile")


@pytest.mark.parametrize("wtype,sessions,rows,d", [("bf16", 32, 8, 1088), ("fp8", 32, 8, 1088),
                                                    ("bf16", 64, 5, 1088), ("fp8", 64, 5, 1088),
                                                    ("bf16", 32, 8, 832), ("bf16", 50, 10, 832),
                                                    ("bf16", 32, 8, 1024)])
def test_bias_and_weight_scales_on_whole_tiles(wtype, sessions, rows, d):
    # 256 or 320 rows fill their row tile, so every n-tile but the last lies
    # wholly inside z: the cloud epilogue's straight-line form adds the bias
    # (and, for E4M3 weights, multiplies by the row scale) once per column.
    # bf16 on 256-row tiles runs one wave per SIMD: 16 K steps (d = 1088)
    # take two weight stages, 12 (d = 832) three, whose ragged tiles read
    # the bias ids from global memory (500 rows: a ragged row tile too);
    # 15 steps (d = 1024) take the two-wave kernel
    cfg = Config(f"whole_tiles_{wtype}_{sessions * rows}_{d}", 37, d=d, d_end=64, vocab=6000,
                 n_sub=3001, subset_kind="choice", sessions=sessions, rows_per_session=rows,
                 wtype=wtype, with_bias=True)
    run_greedy_case(make_workload(cfg), tag=f"bias, {wtype}, {sessions * rows} rows, d = {d}")


def test_fp8_cloud_partial_dense_k_not_multiple_of_64():
    # d_cloud = 1040: the fp8 codes are widened on their way into LDS instead
    # of being copied there directly
    cfg = Config("fp8_dense_k", 28, d=1072, d_end=32, vocab=5000, n_sub=2999, subset_kind="choice",
                 sessions=13, rows_per_session=3, wtype="fp8")
    run_greedy_case(make_workload(cfg), tag="fp8 dense, K % 64 = 16")


# ---------------------------------------------------------------------------
# edge cases of the interface
# ---------------------------------------------------------------------------

def test_k_zero_and_empty_batch():
    cfg = Config("k0", 24, d=128, d_end=16, vocab=700, n_sub=300, subset_kind="choice",
                 sessions=3, rows_per_session=1)
    stats, (q, s, z, tok, acc, f) = run_greedy_case(make_workload(cfg), tag="k=0")
    assert (acc == 0).all()
    dw = P.DeviceWorkload(make_workload(cfg))
    say("[gpu] empty batch")
    q0, s0, _ = sph.cloud_partial(dw.h[:0, 16:], dw.w_cloud, dw.subset, 30.0)
    t0, a0, _ = sph.fuse_verify(q0, s0, dw.h[:0, :16], dw.w_end, dw.subset, 0, 1, None)
    torch.cuda.synchronize()
    assert q0.shape == (0, 300) and t0.shape == (0,) and a0.shape == (0,)


def test_workspace_and_alignment_errors():
    cfg = Config("err", 25, d=128, d_end=16, vocab=700, n_sub=300, subset_kind="choice",
                 sessions=1, rows_per_session=3)
    dw = P.DeviceWorkload(make_workload(cfg))
    say("[gpu] error paths")
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(sph.SphError) as e:
        sph.cloud_partial(dw.h[:, 16:], dw.w_cloud, dw.subset, 30.0, workspace=small)
    assert e.value.code == _lib.SPH_E_WORKSPACE
    with pytest.raises(sph.SphError) as e:
        sph.cloud_partial(dw.h[:, 16:], dw.w_cloud.view(-1)[1:1 + 699 * 112].view(699, 112),
                          dw.subset, 30.0)
    assert e.value.code == _lib.SPH_E_UNSUPPORTED


def test_repeat_runs_are_bit_identical():
    wl = make_workload(CONFIGS["tiny"])
    dw = P.DeviceWorkload(wl)
    say("[gpu] determinism")
    outs = []
    for _ in range(3):
        q, s, z = dw.cloud()
        tok, acc, f = dw.fuse(q, s, np.zeros((1, 2), np.int32))
        torch.cuda.synchronize()
        outs.append([P.host(x) for x in (q, s, z, tok, acc, f)])
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("M", [5, 20])
def test_stale_workspace_contents_are_never_read(M):
    # Poisoned workspaces (huge values / max keys) must not change any result.
    cfg = Config("poison", 26, d=4104, d_end=520, vocab=6000, n_sub=4097, subset_kind="choice",
                 sessions=M // 5, rows_per_session=5)
    wl = make_workload(cfg)
    dw = P.DeviceWorkload(wl)
    say(f"[gpu] poisoned workspace M={M}")
    ref_c = sph.cloud_partial(dw.h[:, 520:], dw.w_cloud, dw.subset, 30.0, want_z=True,
                              workspace=torch.zeros(sph.cloud_partial_workspace(M, dw.subset),
                                                    dtype=torch.uint8, device="cuda"))
    drafts = torch.zeros((cfg.sessions, cfg.k), dtype=torch.int32, device="cuda")
    ref_f = sph.fuse_verify(ref_c[0], ref_c[1], dw.h[:, :520], dw.w_end, dw.subset, cfg.sessions, 5,
                            drafts, workspace=torch.zeros(sph.fuse_verify_workspace(M, dw.subset),
                                                          dtype=torch.uint8, device="cuda"))
    for fill in (0x7F, 0xFF):
        wc = torch.full((sph.cloud_partial_workspace(M, dw.subset),), fill, dtype=torch.uint8, device="cuda")
        wf = torch.full((sph.fuse_verify_workspace(M, dw.subset),), fill, dtype=torch.uint8, device="cuda")
        got_c = sph.cloud_partial(dw.h[:, 520:], dw.w_cloud, dw.subset, 30.0, want_z=True, workspace=wc)
        got_f = sph.fuse_verify(got_c[0], got_c[1], dw.h[:, :520], dw.w_end, dw.subset, cfg.sessions, 5,
                                drafts, workspace=wf)
        torch.cuda.synchronize()
        for a, b in zip(list(ref_c) + list(ref_f[:2]), list(got_c) + list(got_f[:2])):
            np.testing.assert_array_equal(P.host(a), P.host(b))
