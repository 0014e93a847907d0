"""GPU parity of the sampling path (SPH_SAMPLE) against the CPU oracle.

Stage D feeds the GPU's own fused logits to the oracle's sampler: with the
same inputs both sides compute the softmax weights, the nucleus cut and the
inverse CDF in fp64, so tokens must agree except on rows whose recorded
distance to a decision boundary (nucleus cut or CDF interval edge) is below
EPS.  EPS = 1e-9 of the row's probability mass: an fp64 sum of at most 2^18
weights is accurate to ~3e-11 relative, and fp64 exp to ~1e-16.  Stage E
compares with the whole oracle pipeline; there the fused logits differ by
the measured max |df| (stage D), which moves each weight by at most a
factor exp(|df| / tau), so rows closer than 4|df|/tau + EPS are exempt.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_13093_amd as sph
from synth import CONFIGS, Config, make_drafts, make_workload, scale_rows_bf16

import parity as P

pytestmark = pytest.mark.gpu
EPS = 1e-9


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _exempt(info, extra=0.0):
    return (info["cut_margin"] <= EPS + extra) | (info["cdf_margin"] <= EPS + extra)


def run_sample_case(wl, sessions=None, tag="", h_bits=None):
    cfg = wl.cfg
    R = cfg.rows_per_session
    h_bits = wl.h_bits if h_bits is None else h_bits
    sess = np.arange(cfg.sessions) if sessions is None else np.asarray(sessions)
    rows = (sess[:, None] * R + np.arange(R)[None, :]).ravel()

    # oracle pipeline on the checked rows
    orc = oracle.cloud_call(h_bits[rows], cfg.d_end, wl.subset, cfg.clip_c,
                            w_cloud_bits=wl.w_cloud_bits, w_cloud_codes=wl.w_cloud_codes,
                            w_cloud_scale=wl.w_cloud_scale, bias=wl.bias, with_abs=True)
    z_e, absdot_e = oracle.endpoint_partial_logits(h_bits[rows], cfg.d_end, wl.subset,
                                                   wl.w_end_bits, with_abs=True)
    f_orc = oracle.fuse_masked(orc["q"], orc["scale"], z_e)
    # the sampler's counters are (row in session, session): pass the global session ids
    tok_orc, info_orc = _sample_rows(f_orc, wl.subset, cfg, rows)
    ref_tok = np.zeros(cfg.M, np.int32)
    ref_tok[rows] = tok_orc
    drafts = make_drafts(cfg, ref_tok, wl.subset) if cfg.k else None

    say(f"[gpu] {tag or cfg.name}: sample M={cfg.M} n={len(wl.subset)} tau={cfg.temperature} "
        f"top_p={cfg.top_p} wtype={cfg.wtype}")
    dw = P.DeviceWorkload(wl, h_bits=h_bits)
    q, s, z = dw.cloud()
    tok, acc, f = dw.fuse(q, s, drafts)
    torch.cuda.synchronize()
    qh, sh, zh = P.host(q)[rows], P.host(s)[rows], P.host(z)[rows]
    th, ah, fh = P.host(tok), P.host(acc), P.host(f)

    stats = {"A": P.stage_a(zh, orc)}
    P.stage_b(zh, qh, sh, cfg.clip_c)
    stats["C"] = P.stage_c(qh, sh, orc)

    # D: fused logits within tolerance; the oracle's sampler on the GPU's own f
    f_ref = oracle.fuse_masked(qh, sh, z_e)
    df = np.abs(fh[rows].astype(np.float64) - f_ref.astype(np.float64))
    assert (df <= P.tol_of(absdot_e) + P.ULP * np.abs(f_ref)).all(), "stage D: fused logits"
    assert np.all(np.isin(th, wl.subset)), "token outside the subset"
    tok_d, info_d = _sample_rows(fh[rows], wl.subset, cfg, rows)
    ex_d = _exempt(info_d)
    bad = (th[rows] != tok_d) & ~ex_d
    assert not bad.any(), f"stage D: {bad.sum()} sampled tokens differ (rows {rows[bad][:8]})"
    P.check_boundary_rows(th[rows], tok_d, fh[rows], wl.subset, cfg, rows, EPS)
    # accept lengths from the GPU's tokens (exact integer rule)
    acc_ref = oracle.accept_lengths(th, drafts, cfg.sessions, R)
    np.testing.assert_array_equal(ah, acc_ref)

    # E: whole pipelines
    extra = 4.0 * float(np.max(np.abs(fh[rows].astype(np.float64) - f_orc.astype(np.float64)),
                               initial=0.0)) / float(np.float32(cfg.temperature))
    ex_e = _exempt(info_orc, extra)
    bad_e = (th[rows] != tok_orc) & ~ex_e
    assert not bad_e.any(), f"stage E: {bad_e.sum()} tokens differ"
    check_in_perturbed_nucleus(th[rows], tok_orc, f_orc, wl.subset, cfg, extra)
    stats["D"] = {"rows": len(rows), "exempt": int(ex_d.sum()),
                  "mismatch": int((th[rows] != tok_d).sum()),
                  "nucleus_mean": float(np.mean(info_d["nucleus"]))}
    stats["E"] = {"exempt": int(ex_e.sum()), "mismatch": int((th[rows] != tok_orc).sum()),
                  "df_max": float(df.max(initial=0.0))}
    say(f"[gpu] {tag or cfg.name}: ok {stats}")
    return stats, th, fh


def check_in_perturbed_nucleus(tok_gpu, tok_ref, f_ref, subset, cfg, margin):
    """Stage E: where the two pipelines' fused logits differ by up to d, every
    weight moves by at most a factor exp(d / tau) = exp(margin / 4) and so
    does the normaliser, so each probability by at most r = exp(margin / 2).
    A token the GPU may sample lies in its nucleus: the GPU mass of the tokens
    it ranks above is below top_p.  Every token whose oracle probability
    exceeds the GPU token's by the factor r^2 is ranked above it on the GPU,
    with a GPU mass no smaller than its oracle mass over r, so that mass over
    r must be below top_p."""
    diff = np.flatnonzero(tok_gpu != tok_ref)
    if diff.size == 0 or cfg.top_p >= 1.0:
        return
    tau = float(np.float32(cfg.temperature))
    r = np.exp(margin / 2.0)
    subset = np.asarray(subset)
    for m in diff:
        x = f_ref[m].astype(np.float64)
        p = np.exp((x - x.max()) / tau)
        p /= p.sum()
        pt = p[np.searchsorted(subset, tok_gpu[m])]
        above = p[p > pt * r * r].sum() / r
        assert above < float(np.float32(cfg.top_p)), (
            f"stage E row {m}: token {tok_gpu[m]} lies outside the perturbed nucleus")


def _sample_rows(f, subset, cfg, rows):
    """Oracle sampler on selected rows, each with its global row counter."""
    return oracle.sample_select(f, subset, cfg.temperature, cfg.top_p, cfg.philox_seed,
                                cfg.rows_per_session, row_index=rows)


# ---------------------------------------------------------------------------

def test_sample_fp8_workload():
    # the full 640-row launch; the oracle checks 6 whole sessions end to end
    run_sample_case(make_workload(CONFIGS["sample_fp8"]), sessions=[0, 1, 40, 77, 126, 127])


SMALL = [
    # (sessions, R, d, d_end, V, n, tau, top_p, wtype)
    (1, 3, 256, 32, 2000, 1, 0.7, 0.9, "bf16"),         # one-id subset
    (2, 3, 256, 32, 2000, 7, 0.7, 0.9, "bf16"),
    (3, 5, 520, 40, 5000, 4001, 0.7, 0.9, "bf16"),      # ragged chunks per thread
    (2, 4, 1056, 32, 30000, 20000, 1.3, 0.5, "fp8"),    # fp8 weights, 8 rows (skinny)
    (4, 5, 1032, 8, 80000, 70001, 0.7, 0.9, "bf16"),    # n > 65536: values re-read per pass
    (3, 4, 264, 0, 4000, 3001, 0.2, 1.0, "bf16"),       # top_p = 1: whole subset, d_end = 0
    (5, 3, 520, 40, 9000, 8191, 2.0, 0.999, "bf16"),    # 15 rows: MFMA projection
]


@pytest.mark.parametrize("shape", SMALL, ids=[f"S{a}R{b}n{f}t{g}p{h}{w}" for a, b, c, d, e, f, g, h, w in SMALL])
def test_sample_shapes(shape):
    S, R, d, de, V, n, tau, tp, wt = shape
    cfg = Config("sample_small", 40 + S + R + n % 97, d=d, d_end=de, vocab=V, n_sub=n,
                 subset_kind="choice", sessions=S, rows_per_session=R, wtype=wt, mode="sample",
                 temperature=tau, top_p=tp, philox_seed=0x1234_5678_9ABC_DEF0 + n)
    run_sample_case(make_workload(cfg), tag=f"sample {shape}")


def test_sample_ties_at_the_nucleus_cut():
    # all-zero rows: every fused logit is 0, so all weights tie; top_p = 0.9005
    # of 1000 ids keeps exactly the first 901 ids (in id order) and samples
    # uniformly among them
    cfg = Config("ties", 50, d=128, d_end=16, vocab=3000, n_sub=1000, subset_kind="choice",
                 sessions=40, rows_per_session=2, mode="sample", temperature=0.7, top_p=0.9005,
                 philox_seed=99)
    wl = make_workload(cfg)
    h = wl.h_bits.copy()
    h[:] = 0
    stats, tok, f = run_sample_case(wl, h_bits=h, tag="ties")
    assert not f.any()
    pos = np.searchsorted(wl.subset, tok)
    assert pos.max() <= 900 and stats["D"]["exempt"] == 0


def test_sample_many_ties_radix_path():
    # 5000 all-zero logits: the cut lies among more tied elements than are
    # ranked directly, so the key radix select and the tie position decide;
    # top_p = 0.9005 (0.90049999952 in fp32) keeps the first 4503 ids
    cfg = Config("ties_many", 52, d=128, d_end=16, vocab=12000, n_sub=5000, subset_kind="choice",
                 sessions=6, rows_per_session=2, mode="sample", temperature=0.7, top_p=0.9005,
                 philox_seed=101)
    wl = make_workload(cfg)
    h = np.zeros_like(wl.h_bits)
    stats, tok, f = run_sample_case(wl, h_bits=h, tag="ties (radix path)")
    pos = np.searchsorted(wl.subset, tok)
    assert pos.max() <= 4502 and stats["D"]["exempt"] == 0


def test_sample_narrow_rows_radix_path():
    # h scaled by 1e-4: every row's logits span far less than one value
    # bucket ((max - min) / tau < 40 / 4096), so thousands of distinct keys
    # share the cut bucket and the radix select over keys decides
    cfg = Config("narrow", 53, d=256, d_end=32, vocab=9000, n_sub=6000, subset_kind="choice",
                 sessions=4, rows_per_session=3, mode="sample", temperature=0.7, top_p=0.9,
                 philox_seed=202)
    wl = make_workload(cfg)
    h = scale_rows_bf16(wl.h_bits, np.arange(cfg.M), 1e-4)
    stats, tok, f = run_sample_case(wl, h_bits=h, tag="narrow rows (radix path)")
    spread = (f.max(axis=1).astype(np.float64) - f.min(axis=1)) / np.float32(cfg.temperature)
    assert (spread < 0.9 * 40.0 / 4096).all(), spread.max()
    assert len(np.unique(f[0])) > 1024


def test_sample_top_p_to_zero_is_greedy():
    cfg = Config("greedy_limit", 51, d=512, d_end=64, vocab=8192, n_sub=4096, subset_kind="perm",
                 sessions=4, rows_per_session=3, mode="sample", temperature=0.7, top_p=1e-7,
                 philox_seed=7)
    wl = make_workload(cfg)
    stats, tok, f = run_sample_case(wl, tag="top_p -> 0")
    g, _, _ = oracle.greedy_select(f, wl.subset)
    np.testing.assert_array_equal(tok, g)


def test_sample_repeat_runs_are_identical():
    cfg = CONFIGS["tiny"].replace(name="tiny_sample", mode="sample", temperature=0.7, top_p=0.9,
                                  philox_seed=5)
    wl = make_workload(cfg)
    dw = P.DeviceWorkload(wl)
    say("[gpu] sampling determinism")
    outs = []
    for _ in range(3):
        q, s, z = dw.cloud()
        tok, acc, f = dw.fuse(q, s, np.zeros((1, 2), np.int32))
        torch.cuda.synchronize()
        outs.append((P.host(tok), P.host(acc)))
    for o in outs[1:]:
        np.testing.assert_array_equal(o[0], outs[0][0])
        np.testing.assert_array_equal(o[1], outs[0][1])
