"""Host-side logic that needs no GPU: the input generator's helpers and the
benchmark's bookkeeping."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

from synth import Config, make_workload, with_subset

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_with_subset_equals_a_fresh_draw():
    a = Config("a", 7, d=264, d_end=8, vocab=3000, n_sub=3000, subset_kind="full",
               sessions=3, rows_per_session=4)
    b = a.replace(name="b", n_sub=777, subset_kind="choice")
    wa = make_workload(a)
    wb = with_subset(wa, b)
    ref = make_workload(b)
    for k in ("h_bits", "w_end_bits", "w_cloud_bits", "subset"):
        np.testing.assert_array_equal(getattr(wb, k), getattr(ref, k))
    assert wb.full_vocab is False and wb.cfg is b


def test_with_subset_refuses_other_inputs():
    a = Config("a", 7, d=264, d_end=8, vocab=3000, n_sub=3000, subset_kind="full",
               sessions=3, rows_per_session=4)
    wa = make_workload(a)
    with pytest.raises(ValueError):
        with_subset(wa, a.replace(seed_index=8))
    with pytest.raises(ValueError):
        with_subset(wa, a.replace(d_end=16))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_bench_algorithmic_work_matches_the_hand_counts():
    # bytes of one cloud launch: every gathered weight row once (d_cloud
    # weights, 2 bytes bf16 / 1 byte e4m3), its 4-byte id, an fp32 row scale for
    # e4m3 weights, and the M rows of h_cloud; flops 2 M |S| d_cloud.  Counted by
    # hand for the decode, batched and sampling workloads.
    sys.path.insert(0, ROOT)
    import bench
    from synth import CONFIGS
    dec = CONFIGS["decode"]       # 49152 ids x (3840*2 + 4) + 5 x 3840 x 2
    assert bench.algorithmic_bytes(dec, 49152) == 49152 * 7684 + 38400 == 377722368
    bat = CONFIGS["batched"]      # 60000 x (3584*2 + 4) + 320 x 3584 x 2
    assert bench.algorithmic_bytes(bat, 60000) == 430320000 + 2293760
    smp = CONFIGS["sample_fp8"]   # 65536 x (4800 + 4 + 4) + 640 x 4800 x 2
    assert bench.algorithmic_bytes(smp, 65536) == 65536 * 4808 + 6144000
    assert bench.dtype_of(smp) != "bf16" and bench.dtype_of(dec) == "bf16"
