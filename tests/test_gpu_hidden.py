"""GPU parity of the hidden-state codes (Section 5.3 with the Q_b of eq. 18)
and of the endpoint call on them (eq. 11 on the dequantised hidden state).

sph_hidden_quantize must give the oracle's int8 codes and row scales bit for
bit (both sides use a correctly rounded fp32 division and round half to
even).  sph_fuse_verify_hq is checked like stage D of tests/parity.py: the
oracle's endpoint partial on the GPU's own codes (fp64, one rounding) fused
with the GPU's own payload gives fused logits within |df| <= 1e-3 *
sum |q s w| + 1e-5 + ulp, and tokens equal unless a competitor lies within
the elementwise bound; accept lengths follow exactly.  Shapes cover both
skinny row groups, the register-staged MFMA kernel (d_end not a multiple of
64) and the 128-, 256- and 320-row direct-to-LDS tiles.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_13093_amd as sph
from synth import CONFIGS, Config, make_drafts, make_workload

import parity as P

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


HQ_SHAPES = [
    # (M, d, ldh): bf16 rows, the first d columns of rows ldh apart
    (1, 256, 256),
    (5, 4096, 4096),     # register path (d <= 8192, multiple of 8, aligned)
    (7, 4100, 4104),     # d not a multiple of 8: two-pass path
    (3, 9000, 9000),     # d > 8192: two-pass path
    (600, 512, 4096),    # strided view of the first 512 columns
    (2, 0, 8),           # no columns: scales 0
]


@pytest.mark.parametrize("shape", HQ_SHAPES, ids=[f"M{m}d{d}ld{l}" for m, d, l in HQ_SHAPES])
def test_hidden_quantize_bit_exact(shape):
    M, d, ldh = shape
    rng = np.random.default_rng(1000 + M + d)
    x = (rng.standard_normal((M, ldh)) * rng.uniform(0.05, 30.0, (M, 1))).astype(np.float32)
    if M >= 3 and d > 10:
        x[1, :] = 0.0                  # a zero row
        x[2, d // 2] = -500.0          # an outlier sets its row's scale
        x[0, :8] = [127, -1.5, 2.5, 0.25, -127, 3.5, -0.5, 126.5]
        x[0, 8:] = 0.0                 # s = 1 for row 0: codes are rint(x), ties to even
    from synth import f32_to_bf16_bits
    hb = f32_to_bf16_bits(x)
    q_ref, s_ref = oracle.hidden_quantize(hb[:, :d])
    say(f"[gpu] hidden_quantize M={M} d={d} ldh={ldh}")
    h = P.to_dev(hb, torch.bfloat16)
    hq, hs = sph.hidden_quantize(h[:, :d])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(hs).view(np.uint32), s_ref.view(np.uint32))
    np.testing.assert_array_equal(P.host(hq), q_ref)


def run_hq_case(wl, tag, bits=8, block=0, sessions=None):
    cfg = wl.cfg
    R = cfg.rows_per_session
    S_all = cfg.sessions
    sess = np.arange(S_all) if sessions is None else np.asarray(sessions)
    rows = (sess[:, None] * R + np.arange(R)[None, :]).ravel()
    n = len(wl.subset)

    # the cloud returns the whole hidden row as codes; the endpoint uses its first d_end
    hq_ref, hs_ref = oracle.hidden_quantize(wl.h_bits)
    z_e_orc, _ = oracle.endpoint_partial_logits_hq(hq_ref[rows], hs_ref[rows], cfg.d_end,
                                                   wl.subset, wl.w_end_bits)
    orc = oracle.cloud_call(wl.h_bits[rows], cfg.d_end, wl.subset, cfg.clip_c,
                            w_cloud_bits=wl.w_cloud_bits, w_cloud_codes=wl.w_cloud_codes,
                            w_cloud_scale=wl.w_cloud_scale, bias=wl.bias)
    fmt = oracle.clip_quantize_fmt(orc["z"], cfg.clip_c, bits, block)
    f_orc = oracle.fuse_masked_fmt(fmt["q"], fmt["scale"], z_e_orc, block)
    ref_tok = np.zeros(cfg.M, np.int32)
    ref_tok[rows] = oracle.greedy_select(f_orc, wl.subset)[0]
    drafts_all = make_drafts(cfg, ref_tok, wl.subset) if cfg.k else None

    say(f"[gpu] {tag}: M={cfg.M} d={cfg.d} d_end={cfg.d_end} n={n} bits={bits} block={block}")
    dw = P.DeviceWorkload(wl)
    q, s, z = dw.cloud(bits=bits, block=block)
    hq, hs = sph.hidden_quantize(dw.h)
    d = None if drafts_all is None else P.to_dev(np.asarray(drafts_all, np.int32))
    mode = sph.GREEDY if cfg.mode == "greedy" else sph.SAMPLE
    tok, acc, f = sph.fuse_verify_hq(q, s, hq, hs, cfg.d_end, dw.w_end, dw.subset, S_all, R, d,
                                     mode=mode, temperature=cfg.temperature, top_p=cfg.top_p,
                                     seed=cfg.philox_seed, want_fused=True, bits=bits, block=block)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(hq), hq_ref, err_msg="hidden codes")
    np.testing.assert_array_equal(P.host(hs).view(np.uint32), hs_ref.view(np.uint32))
    qh, sh, zh = P.host(q)[rows], P.host(s)[rows], P.host(z)[rows]
    codes = P.stage_b_fmt(zh, qh.view(np.uint8), sh, cfg.clip_c, bits, block)
    th, ah, fh = P.host(tok), P.host(acc), P.host(f)[rows]

    # D: the oracle's endpoint steps on the GPU's codes and payload
    z_e, absdot = oracle.endpoint_partial_logits_hq(P.host(hq)[rows], P.host(hs)[rows],
                                                    cfg.d_end, wl.subset, wl.w_end_bits,
                                                    with_abs=True)
    f_ref = oracle.fuse_masked_fmt(codes, sh.reshape(len(rows), -1), z_e, block)
    bound = P.tol_of(absdot) + P.ULP * np.abs(f_ref.astype(np.float64))
    df = np.abs(fh.astype(np.float64) - f_ref.astype(np.float64))
    assert (df <= bound).all(), f"fused logits outside tolerance, worst {df.max():.3e}"
    assert np.all(np.isin(th, wl.subset)), "token outside the subset"
    if cfg.mode == "greedy":
        tok_ref = oracle.greedy_select(f_ref, wl.subset)[0]
        drafts = drafts_all[sess] if cfg.k else None
        acc_ref = oracle.accept_lengths(tok_ref, drafts, len(sess), R)
        ex = P.exempt_rows(f_ref, bound)
        st = P.check_tokens_and_accept(th[rows], ah[sess], tok_ref, acc_ref, ex, wl.subset,
                                       len(sess), R, f_ref, bound, drafts)
    else:
        tok_ref, info = oracle.sample_select(fh, wl.subset, cfg.temperature, cfg.top_p,
                                             cfg.philox_seed, R, row_index=rows)
        ex = (info["cut_margin"] <= 1e-9) | (info["cdf_margin"] <= 1e-9)
        bad = (th[rows] != tok_ref) & ~ex
        assert not bad.any(), f"{bad.sum()} sampled tokens differ"
        P.check_boundary_rows(th[rows], tok_ref, fh, wl.subset, cfg, rows, 1e-9)
        np.testing.assert_array_equal(ah, oracle.accept_lengths(th, drafts_all, S_all, R))
        st = {"exempt": int(ex.sum())}
    say(f"[gpu] {tag}: ok df_max={df.max(initial=0.0):.3e} {st}")


HQ_FUSE = [
    # (sessions, R, d, d_end, V, n)
    (1, 5, 1032, 256, 4000, 2501),   # skinny, d_end = 256
    (13, 1, 1096, 72, 9000, 4097),   # skinny, two row groups
    (3, 3, 520, 40, 3000, 1001),     # 9 rows: register-staged MFMA (d_end % 64 != 0)
    (8, 5, 1032, 128, 4000, 2560),   # 40 rows: 128-row direct-to-LDS tile
    (13, 10, 2056, 512, 9000, 8193), # 130 rows: 256-row tile
    (24, 25, 1096, 128, 9000, 4097), # 600 rows: two 320-row tiles
    (3, 3, 264, 0, 2000, 777),       # d_end = 0: the codes are not read
]


@pytest.mark.parametrize("shape", HQ_FUSE, ids=[f"S{s}R{r}d{d}de{de}V{v}n{n}" for s, r, d, de, v, n in HQ_FUSE])
def test_fuse_verify_on_hidden_codes(shape):
    S, R, d, de, V, n = shape
    cfg = Config("hq", 80 + sum(shape) % 1000, d=d, d_end=de, vocab=V, n_sub=n,
                 subset_kind="choice", sessions=S, rows_per_session=R)
    run_hq_case(make_workload(cfg), f"hq {shape}")


def test_fuse_verify_on_hidden_codes_with_4bit_payload():
    cfg = Config("hq4", 91, d=1096, d_end=128, vocab=9000, n_sub=4097, subset_kind="choice",
                 sessions=24, rows_per_session=5)
    run_hq_case(make_workload(cfg), "hq 120 rows, 4-bit payload", bits=4, block=256)


def test_fuse_verify_on_hidden_codes_sampling():
    cfg = Config("hq_sample", 92, d=520, d_end=40, vocab=9000, n_sub=8191, subset_kind="choice",
                 sessions=5, rows_per_session=3, mode="sample", temperature=0.7, top_p=0.9,
                 philox_seed=0x5EED_0F_C0DE5)
    run_hq_case(make_workload(cfg), "hq sampling")


@pytest.mark.parametrize("name", ["decode", "dense_sub"])
def test_hidden_codes_benchmark_workloads(name):
    sessions = None if name == "decode" else [0, 77, 160, 255]
    run_hq_case(make_workload(CONFIGS[name]), f"{name} on hidden codes", sessions=sessions)
