"""Seeded random configurations through the staged parity checks.

Each case draws a shape (sessions, rows per session, d, d_end, V, |S|) within
the documented limits, a weight type and a payload format, so that the
skinny and MFMA projections, every row tile, ragged tiles on both axes,
bf16 and fp8 weights, every payload format and the hidden-state codes meet
shapes no hand-picked case has.  The checks are those of the format and
hidden-code tests (stages A-E of tests/parity.py)."""

import numpy as np
import pytest

from synth import Config, make_workload

from test_gpu_hidden import run_hq_case
from test_gpu_payload import run_format_case
from test_gpu_sampling import run_sample_case

pytestmark = pytest.mark.gpu

_FORMATS = [(8, 0), (4, 0), (4, 256), (8, 256), (4, 1024), (8, 4096)]


def _draw(i, rng):
    sessions = int(rng.integers(1, 21))
    R = int(rng.integers(1, 10))
    wtype = "fp8" if rng.random() < 0.3 else "bf16"
    step = 16 if wtype == "fp8" else 8
    d_end = int(rng.choice([0, 8, 40, 64, 72, 128, 256, 264, 512]))
    d_cloud = step * int(rng.integers(1, 2048 // step + 1))
    n = int(rng.integers(1, 12001))
    V = n + int(rng.integers(0, 8000))
    bits, block = _FORMATS[int(rng.integers(0, len(_FORMATS)))]
    hq = rng.random() < 0.35
    return dict(i=i, sessions=sessions, R=R, d=d_end + d_cloud, d_end=d_end, V=V, n=n,
                wtype=wtype, bits=bits, block=block, hq=hq)


_RNG = np.random.default_rng(2607)
CASES = [_draw(i, _RNG) for i in range(24)]


def _id(c):
    return (f"{c['i']}-S{c['sessions']}R{c['R']}d{c['d']}de{c['d_end']}n{c['n']}"
            f"-{c['wtype']}-b{c['bits']}k{c['block']}{'-hq' if c['hq'] else ''}")


@pytest.mark.parametrize("c", CASES, ids=[_id(c) for c in CASES])
def test_random_configuration(c):
    cfg = Config("random", 300 + c["i"], d=c["d"], d_end=c["d_end"], vocab=c["V"], n_sub=c["n"],
                 subset_kind="choice", sessions=c["sessions"], rows_per_session=c["R"],
                 wtype=c["wtype"], with_bias=bool(c["i"] % 3 == 0))
    wl = make_workload(cfg)
    if c["hq"]:
        run_hq_case(wl, f"random {_id(c)}", bits=c["bits"], block=c["block"])
    else:
        run_format_case(wl, c["bits"], c["block"], f"random {_id(c)}")


def _draw_sample(i, rng):
    c = _draw(100 + i, rng)
    c["tau"] = float(np.round(rng.uniform(0.2, 2.0), 3))
    c["top_p"] = float(np.round(rng.choice([rng.uniform(0.05, 0.99), 1.0]), 3))
    return c


_RNG_S = np.random.default_rng(2608)
SAMPLE_CASES = [_draw_sample(i, _RNG_S) for i in range(10)]


@pytest.mark.parametrize("c", SAMPLE_CASES,
                         ids=[f"{c['i']}-S{c['sessions']}R{c['R']}d{c['d']}de{c['d_end']}n{c['n']}-"
                              f"{c['wtype']}-t{c['tau']}-p{c['top_p']}" for c in SAMPLE_CASES])
def test_random_sampling_configuration(c):
    cfg = Config("random_sample", 500 + c["i"], d=c["d"], d_end=c["d_end"], vocab=c["V"],
                 n_sub=c["n"], subset_kind="choice", sessions=c["sessions"],
                 rows_per_session=c["R"], wtype=c["wtype"], mode="sample",
                 temperature=c["tau"], top_p=c["top_p"],
                 philox_seed=0x2607_1309_0000_0000 + c["i"])
    run_sample_case(make_workload(cfg), tag=f"random sample {c['i']}")


def _draw_one_wave(i, rng):
    """bf16 shapes that the one-wave cloud kernel takes: 256-row tiles (129 to
    256 rows, or 321 to 512) and an even number of 64-wide K steps, a multiple
    of 6 in half of the cases (three weight stages)."""
    while True:
        sessions = int(rng.integers(8, 65))
        R = int(rng.integers(4, 9))
        M = sessions * R
        if 129 <= M <= 256 or 321 <= M <= 512:
            break
    steps = int(rng.choice([6, 12, 18, 24])) if i % 2 == 0 else int(rng.choice([2, 4, 8, 10, 14, 16]))
    d_end = int(rng.choice([0, 64, 128]))
    n = int(rng.integers(1, 6001))
    V = n + int(rng.integers(0, 4000))
    bits, block = _FORMATS[int(rng.integers(0, 2))]  # per-row scales: the cloud kernel writes z
    return dict(i=i, sessions=sessions, R=R, d=d_end + 64 * steps, d_end=d_end, V=V, n=n,
                wtype="bf16", bits=bits, block=block, hq=False)


_RNG_W = np.random.default_rng(2609)
ONE_WAVE_CASES = [_draw_one_wave(i, _RNG_W) for i in range(10)]


@pytest.mark.parametrize("c", ONE_WAVE_CASES, ids=[_id(c) for c in ONE_WAVE_CASES])
def test_one_wave_cloud_configuration(c):
    cfg = Config("random_one_wave", 700 + c["i"], d=c["d"], d_end=c["d_end"], vocab=c["V"],
                 n_sub=c["n"], subset_kind="choice", sessions=c["sessions"], rows_per_session=c["R"],
                 wtype="bf16", with_bias=bool(c["i"] % 3 == 1))
    run_format_case(make_workload(cfg), c["bits"], c["block"], f"one-wave {_id(c)}")
