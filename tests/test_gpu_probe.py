"""The measurement helpers of include/sph_probe.h run on the device and
report a plausible operation count (they compute nothing the method uses)."""

import pytest
import torch

import paper_2607_13093_amd as sph

pytestmark = pytest.mark.gpu


def test_probe_read_runs():
    dev = torch.device("cuda:0")
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    for nbytes in (16, 16 * 1000, 64 << 20):   # one chunk, a ragged grid, many blocks
        buf = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        sph.probe_read(buf, sink)
    torch.cuda.synchronize()


def test_probe_mfma_counts_flops():
    dev = torch.device("cuda:0")
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    flops = sph.probe_mfma(10, sink)
    torch.cuda.synchronize()
    # 256 workgroups x 4 waves x 10 iterations x 32 MFMAs x (2*32*32*16)
    assert flops == 256 * 4 * 10 * 32 * 2 * 32 * 32 * 16
