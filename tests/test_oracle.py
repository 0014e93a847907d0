"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names what fixes the expected value: a hand-worked example, a
library routine for a special case, a closed form, an invariant, published
known-answer vectors, exact rational arithmetic, or a statistical law.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from synth import (Config, f32_to_bf16_bits, make_workload, plant_masked_supertoken,
                   scale_rows_bf16)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bits(a):
    return f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


# ---------------------------------------------------------------------------
# input decodings vs library conversions
# ---------------------------------------------------------------------------

def test_bf16_decode_matches_torch_on_every_pattern():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = oracle.decode_bf16(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().double().numpy()
    np.testing.assert_array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(ours[ok], ref[ok])


def test_e4m3_decode_matches_torch_on_all_256_codes():
    codes = np.arange(256, dtype=np.uint8)
    ours = oracle.decode_e4m3(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().double().numpy()
    np.testing.assert_array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(ours[ok], ref[ok])
    assert np.nanmax(ours) == 448.0 and np.isnan(ours).sum() == 2


def test_generator_bf16_rounding_matches_torch():
    x = np.random.default_rng(7).standard_normal(100000).astype(np.float32) * 3
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(f32_to_bf16_bits(x), ref)


# ---------------------------------------------------------------------------
# Philox4x32-10
# ---------------------------------------------------------------------------

# Known-answer vectors published with the Random123 implementation of
# Philox4x32-10 (Salmon et al., SC'11): (counter, key) -> output.
PHILOX_KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,out", PHILOX_KAT)
def test_philox_known_answers(ctr, key, out):
    assert oracle.philox4x32_10(ctr, key) == out


def test_philox_uniform_is_uniform():
    from scipy import stats
    u = np.array([oracle.philox_uniform(0x1234_5678_9ABC_DEF0, r, s)
                  for s in range(400) for r in range(10)])
    assert u.min() >= 0 and u.max() < 1
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    assert np.all(u * 2 ** 24 == np.floor(u * 2 ** 24))  # 24-bit grid


# ---------------------------------------------------------------------------
# the hand-worked example (golden fixture)
# ---------------------------------------------------------------------------

def test_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    W = np.array(g["weights_by_id"], dtype=np.float32)
    H = np.array(g["h"], dtype=np.float32)
    S = np.array(g["subset"], dtype=np.int32)
    de = g["d_end"]
    wb, hb = _bits(W), _bits(H)
    w_end, w_cloud = np.ascontiguousarray(wb[:, :de]), np.ascontiguousarray(wb[:, de:])

    cl = oracle.cloud_call(hb, de, S, g["clip_c"], w_cloud_bits=w_cloud)
    np.testing.assert_array_equal(cl["z"], np.array(g["z_cloud"], np.float32))
    np.testing.assert_array_equal(cl["y"], np.array(g["y"], np.float32))
    np.testing.assert_array_equal(cl["amax"], np.array(g["amax"], np.float32))
    np.testing.assert_array_equal(cl["scale"], np.full(3, np.float32(30.0) / np.float32(127.0)))
    np.testing.assert_array_equal(cl["q"], np.array(g["q"], np.int8))

    z_e, _ = oracle.endpoint_partial_logits(hb, de, S, w_end)
    np.testing.assert_array_equal(z_e, np.array(g["z_end"], np.float32))

    # eq. 9 on the masked ids: they dominate the unmasked head
    full = oracle.full_head_logits(hb, W.astype(np.float64))
    np.testing.assert_array_equal(full[:, g["full_head_masked_ids"]["ids"]],
                                  np.array(g["full_head_masked_ids"]["logits"], np.float64))

    f = oracle.fuse_masked(cl["q"], cl["scale"], z_e)
    exact = np.array(g["fused_exact_numerators_over_127"], np.float64) / 127.0
    # s is the fp32 nearest to 30/127: |q| * |s - 30/127| <= 127 * 2^-26
    np.testing.assert_allclose(f, exact, rtol=0, atol=4e-6)

    tok, _, _ = oracle.greedy_select(f, S)
    np.testing.assert_array_equal(tok, g["tokens"])
    for case in g["verify_cases"]:
        a = oracle.accept_lengths(tok, np.array([case["drafts"]]), 1, 3)
        assert a[0] == case["accept"]
        committed = list(case["drafts"][:a[0]]) + [int(tok[a[0]])]
        assert committed == case["committed"]


# ---------------------------------------------------------------------------
# the split identity (eq. 9-13) and special cases that are library routines
# ---------------------------------------------------------------------------

def _small(seed, d=96, d_end=24, V=500, n=200, M=7, bias=True):
    rng = np.random.default_rng(seed)
    H = _bits(rng.standard_normal((M, d)))
    W = _bits(rng.standard_normal((V, d)) / np.sqrt(d))
    S = np.sort(rng.choice(V, n, replace=False)).astype(np.int32)
    b = rng.standard_normal(V).astype(np.float32) if bias else None
    return H, W, S, b


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_split_identity_against_unsplit_head(seed):
    H, W, S, b = _small(seed)
    de = 24
    z_c, _ = oracle.cloud_partial_logits(H, de, S, w_cloud_bits=np.ascontiguousarray(W[:, de:]), bias=b)
    z_e, _ = oracle.endpoint_partial_logits(H, de, S, np.ascontiguousarray(W[:, :de]))
    full = oracle.full_head_logits(H, oracle.decode_bf16(W), bias=b)[:, S]
    # each partial is one fp32 rounding of its exact value
    err = np.abs(z_c.astype(np.float64) + z_e.astype(np.float64) - full)
    bound = 2.0 ** -24 * (np.abs(z_c) + np.abs(z_e)) + 1e-30
    assert np.all(err <= bound * 1.0000001)


def test_split_identity_catches_a_swapped_split():
    # the endpoint owns the FIRST d_end dims (eq. 10): swapping the halves breaks the identity
    H, W, S, b = _small(3, bias=False)
    de = 24
    z_c, _ = oracle.cloud_partial_logits(H, de, S, w_cloud_bits=np.ascontiguousarray(W[:, de:]))
    full = oracle.full_head_logits(H, oracle.decode_bf16(W))[:, S]
    wrong, _ = oracle.endpoint_partial_logits(H[:, ::-1].copy(), de, S, np.ascontiguousarray(W[:, :de]))
    assert np.abs(z_c + wrong - full).max() > 1e-2


def test_d_end_zero_is_the_whole_head_via_torch_linear():
    H, W, S, b = _small(4)
    z_c, _ = oracle.cloud_partial_logits(H, 0, S, w_cloud_bits=W, bias=b)
    z_e, _ = oracle.endpoint_partial_logits(H, 0, S, W[:, :0])
    Ht = torch.from_numpy(oracle.decode_bf16(H))
    Wt = torch.from_numpy(oracle.decode_bf16(W[S]))
    ref = torch.nn.functional.linear(Ht, Wt, torch.from_numpy(b[S].astype(np.float64))).float().numpy()
    np.testing.assert_allclose(z_c, ref, rtol=2 ** -23, atol=0)
    assert not z_e.any()


def test_full_vocab_subset_via_torch_linear():
    H, W, _, _ = _small(5, bias=False)
    S = np.arange(W.shape[0], dtype=np.int32)
    de = 24
    z_c, _ = oracle.cloud_partial_logits(H, de, S, w_cloud_bits=np.ascontiguousarray(W[:, de:]))
    ref = torch.nn.functional.linear(torch.from_numpy(oracle.decode_bf16(H[:, de:])),
                                     torch.from_numpy(oracle.decode_bf16(W[:, de:]))).float().numpy()
    np.testing.assert_allclose(z_c, ref, rtol=2 ** -23, atol=0)


def test_fp8_cloud_weights_via_torch_float8():
    H, W, S, _ = _small(6, bias=False)
    from synth import fp8_encode_rows
    de = 24
    codes, scale = fp8_encode_rows(np.ascontiguousarray(W[:, de:]))
    z_c, _ = oracle.cloud_partial_logits(H, de, S, w_cloud_codes=codes, w_cloud_scale=scale)
    Wq = torch.from_numpy(codes).view(torch.float8_e4m3fn).double() * torch.from_numpy(scale).double()[:, None]
    ref = torch.nn.functional.linear(torch.from_numpy(oracle.decode_bf16(H[:, de:])), Wq[S]).float().numpy()
    np.testing.assert_allclose(z_c, ref, rtol=2 ** -23, atol=0)


def test_absdot_bounds_the_dot():
    H, W, S, b = _small(8)
    z, a = oracle.cloud_partial_logits(H, 24, S, w_cloud_bits=np.ascontiguousarray(W[:, 24:]),
                                       bias=b, with_abs=True)
    assert np.all(np.abs(z) <= a * (1 + 2 ** -23))


# ---------------------------------------------------------------------------
# clip + quantise (eq. 18 reading)
# ---------------------------------------------------------------------------

def test_quantizer_invariants():
    rng = np.random.default_rng(11)
    z = (rng.standard_normal((16, 3000)) * rng.uniform(0.1, 20, (16, 1))).astype(np.float32)
    out = oracle.clip_quantize(z, 30.0)
    y, s, q = out["y"], out["scale"], out["q"].astype(np.int32)
    assert np.all(np.abs(y) <= 30)
    assert np.all(np.abs(q) <= 127)
    err = np.abs(q * s[:, None].astype(np.float64) - y.astype(np.float64))
    assert np.all(err <= s[:, None] * (0.5 + 2 ** -20))
    at = np.argmax(np.abs(y), axis=1)
    assert np.all(np.abs(q[np.arange(16), at]) == 127)
    assert np.all(np.sign(q) * np.sign(y) >= 0)


def test_quantizer_rounds_half_to_even():
    # amax = 127 gives s = 1 exactly, so t = y
    z = np.array([[127, 2.5, 3.5, -2.5, -3.5, 0.5, 1.5, 126.5]], dtype=np.float32)
    out = oracle.clip_quantize(z, 300.0)
    assert out["scale"][0] == 1.0
    np.testing.assert_array_equal(out["q"][0], [127, 2, 4, -2, -4, 0, 2, 126])


# ---------------------------------------------------------------------------
# hidden-state quantisation (Section 5.3 with eq. 18) and eq. 11 on it
# ---------------------------------------------------------------------------

def _bf(x):
    return f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def test_hidden_quantize_unit_scale_row():
    # a row whose largest |x| is 127 has s = 1, so the codes are rint(x)
    # (ties to even); a second row of zeros has s = 0 and zero codes
    h = _bf([[127, -1.5, 2.5, 0.25, -127, 3.5, -0.5, 126.5],
             [0, 0, 0, 0, 0, 0, 0, 0]])
    q, s = oracle.hidden_quantize(h)
    assert s[0] == 1.0 and s[1] == 0.0
    np.testing.assert_array_equal(q[0], [127, -2, 2, 0, -127, 4, 0, 126])
    assert not q[1].any()


def test_hidden_quantize_invariants():
    rng = np.random.default_rng(12)
    x = (rng.standard_normal((12, 700)) * rng.uniform(0.01, 50, (12, 1))).astype(np.float32)
    x[3, 17] = 900.0    # an outlier sets its row's scale
    h = _bf(x)
    xv = oracle.decode_bf16(h)
    q, s = oracle.hidden_quantize(h)
    qi = q.astype(np.int32)
    assert np.all(np.abs(qi) <= 127)
    # t = fp32(x / s) is within ulp(t)/2 <= 2^-18 of x / s for |t| < 128,
    # so |q - x/s| <= 1/2 + 2^-18
    err = np.abs(qi * s[:, None].astype(np.float64) - xv)
    assert np.all(err <= s[:, None].astype(np.float64) * (0.5 + 2 ** -18))
    at = np.argmax(np.abs(xv), axis=1)
    assert np.all(np.abs(qi[np.arange(12), at]) == 127)
    assert np.all(np.sign(qi) * np.sign(xv) >= 0)
    assert s[3] == np.float32(np.float32(900.0) / np.float32(127.0))
    # with a clip above every |x| the logit quantiser gives the same codes and scales
    ref = oracle.clip_quantize(xv.astype(np.float32), 1e30)
    np.testing.assert_array_equal(ref["q"], q)
    np.testing.assert_array_equal(ref["scale"], s)


def test_endpoint_partial_hq_hand_example():
    # codes [2, -3] with s = 0.5 are the values [1, -1.5]; ids 0 and 1 of
    # W_end are [1, 1] and [2, -1]: z = [1 - 1.5, 2 + 1.5]; a third code
    # column lies beyond d_end and must not enter the sum
    hq = np.array([[2, -3, 99]], dtype=np.int8)
    w = _bf([[1, 1], [2, -1], [5, 5]])
    z, a = oracle.endpoint_partial_logits_hq(hq, np.array([0.5], np.float32), 2, [0, 1], w,
                                             with_abs=True)
    np.testing.assert_array_equal(z, [[-0.5, 3.5]])
    np.testing.assert_array_equal(a, [[2.5, 3.5]])


def test_endpoint_partial_hq_equals_bf16_partial_when_exact():
    # rows whose dequantised values are bf16 numbers: integers with maximum
    # 127 (s = 1) and integers / 8 with maximum 127 / 8 (s = 2^-3); the
    # endpoint partial on the codes must equal eq. 11 on those values, row
    # by row (two scales in one call)
    rng = np.random.default_rng(13)
    d, d_end = 96, 64
    ints = rng.integers(-127, 128, size=(2, d)).astype(np.float32)
    ints[:, 5] = 127
    x = ints.copy()
    x[1] /= 8
    h = _bf(x)
    q, s = oracle.hidden_quantize(h)
    assert s[0] == 1.0 and s[1] == 0.125
    np.testing.assert_array_equal(q.astype(np.float32), ints)
    w = _bf(rng.standard_normal((300, d_end)).astype(np.float32) / 8)
    S = np.sort(rng.choice(300, 77, replace=False))
    z_hq, _ = oracle.endpoint_partial_logits_hq(q, s, d_end, S, w)
    z_ref, _ = oracle.endpoint_partial_logits(h, d_end, S, w)
    np.testing.assert_array_equal(z_hq, z_ref)


def test_clip_and_zero_rows():
    cfg = Config("t", 0, d=512, d_end=64, vocab=8192, n_sub=4096, subset_kind="perm",
                 sessions=1, rows_per_session=3)
    wl = make_workload(cfg)
    h = scale_rows_bf16(wl.h_bits, [0], 10.0)
    h[2] = 0
    out = oracle.cloud_call(h, 64, wl.subset, 30.0, w_cloud_bits=wl.w_cloud_bits)
    assert np.abs(out["z"][0]).max() > 30          # the scaled row does exceed the clip
    assert out["amax"][0] == 30.0
    assert out["scale"][0] == np.float32(30.0) / np.float32(127.0)
    assert out["amax"][1] < 30                      # an ordinary row is not clipped
    assert out["scale"][2] == 0 and not out["q"][2].any()


# ---------------------------------------------------------------------------
# configurable payload format: b in {4, 8}, one scale per row or per block
# (eq. 18 with a configurable bit width; eq. 21's payload size)
# ---------------------------------------------------------------------------

def test_format_b8_per_row_is_the_int8_reading():
    rng = np.random.default_rng(12)
    z = (rng.standard_normal((7, 1001)) * 6).astype(np.float32)
    a, b = oracle.clip_quantize(z, 30.0), oracle.clip_quantize_fmt(z, 30.0, bits=8, block=0)
    np.testing.assert_array_equal(a["q"], b["q"])
    np.testing.assert_array_equal(a["scale"], b["scale"][:, 0])


@pytest.mark.parametrize("bits,block", [(4, 0), (4, 256), (8, 256), (4, 1024), (8, 4096)])
def test_format_invariants(bits, block):
    rng = np.random.default_rng(13)
    n = 3001                                        # ragged last block, odd for the 4-bit packing
    z = (rng.standard_normal((9, n)) * rng.uniform(0.1, 20, (9, 1))).astype(np.float32)
    out = oracle.clip_quantize_fmt(z, 30.0, bits=bits, block=block)
    y, s, q = out["y"], out["scale"], out["q"].astype(np.int32)
    qmax = 2 ** (bits - 1) - 1
    width = n if block == 0 else block
    cols = np.arange(n) // width
    sc = s[:, cols].astype(np.float64)
    assert np.all(np.abs(q) <= qmax)
    assert np.all(np.abs(q * sc - y) <= sc * (0.5 + 2 ** -20))
    for k in range(s.shape[1]):
        seg = np.abs(y[:, k * width:(k + 1) * width])
        at = np.argmax(seg, axis=1) + k * width
        assert np.all(np.abs(q[np.arange(9), at]) == qmax)
        # a block's scale never exceeds the row's
        assert np.all(s[:, k] <= np.abs(y).max(axis=1) / qmax * (1 + 2 ** -22))
    np.testing.assert_array_equal(oracle.unpack_codes(oracle.pack_codes(out["q"], bits), n, bits), out["q"])
    assert oracle.pack_codes(out["q"], bits).shape[1] == -(-n * bits // 8)
    assert oracle.payload_bytes(n, bits, block) == -(-n * bits // 8) + 4 * s.shape[1]


def test_payload_bytes_pinned_to_eq21():
    # eq. 21 (Section 7.6): codes cost |V_l| * b / 8 bytes; the paper's figure
    # for a full 150,000-entry int8 logit row is about 146.5 KB.  The other
    # cases are counted by hand (tests/golden/payload_eq21.json); the odd
    # lengths and partial blocks fail a floor in place of a ceiling.
    with open(os.path.join(GOLDEN, "payload_eq21.json")) as f:
        g = json.load(f)
    fig = g["paper_figure"]
    codes = oracle.payload_bytes(fig["n"], fig["bits"], 0) - 4
    assert codes == fig["code_bytes"]
    assert round(codes / 1024, 1) == fig["kib_rounded_to_0_1"]
    for c in g["hand_counted"]:
        assert oracle.payload_bytes(c["n"], c["bits"], c["block"]) == c["bytes"], c


def test_format_4bit_worked_example():
    # two blocks of 4 positions, codes in [-7, 7]
    z = np.array([[0.7, -1.4, 0.35, 0.0, 2.0, 3.5, -0.25, 7.0, 1.0]], dtype=np.float32)
    out = oracle.clip_quantize_fmt(z, 30.0, bits=4, block=4)
    # block 0: amax 1.4, s = fp32(1.4/7) = 0.2: t = 3.5, -7, 1.75, 0 -> 4 (half to even), -7, 2, 0
    # block 1: amax 7,   s = 1:               t = 2, 3.5, -0.25, 7 -> 2, 4, 0, 7
    # block 2: amax 1,   s = fp32(1/7):       t = 7                -> 7
    np.testing.assert_array_equal(out["scale"][0], np.float32([np.float32(1.4) / np.float32(7),
                                                               1.0, np.float32(1.0) / np.float32(7)]))
    np.testing.assert_array_equal(out["q"][0], [4, -7, 2, 0, 2, 4, 0, 7, 7])
    # nibbles (two's complement): 4|-7 -> 0x94, 2|0 -> 0x02, 2|4 -> 0x42, 0|7 -> 0x70, 7|pad -> 0x07
    np.testing.assert_array_equal(oracle.pack_codes(out["q"], 4)[0], [0x94, 0x02, 0x42, 0x70, 0x07])
    np.testing.assert_array_equal(oracle.pack_codes([[1, -1, 7, -7]], 4)[0], [0xF1, 0x97])


def test_format_fuse_per_row_equals_fuse_masked_and_uses_block_scales():
    rng = np.random.default_rng(14)
    q = rng.integers(-7, 8, (3, 600)).astype(np.int8)
    s = rng.uniform(0.01, 1, (3, 3)).astype(np.float32)
    ze = rng.standard_normal((3, 600)).astype(np.float32)
    np.testing.assert_array_equal(oracle.fuse_masked_fmt(q, s[:, :1], ze, 0), oracle.fuse_masked(q, s[:, 0], ze))
    f = oracle.fuse_masked_fmt(q, s, ze, 256)
    j = 513                                         # third block
    assert f[1, j] == np.float32(float(q[1, j]) * float(s[1, 2]) + float(ze[1, j]))
    # hand example: unit codes, zero partials, blocks of 2 with scales 1, 2, 4
    # (the last block holds one position)
    f = oracle.fuse_masked_fmt(np.ones((1, 5), np.int8), np.float32([[1, 2, 4]]),
                               np.zeros((1, 5), np.float32), 2)
    np.testing.assert_array_equal(f[0], [1, 1, 2, 2, 4])


# ---------------------------------------------------------------------------
# fusion rounding
# ---------------------------------------------------------------------------

def _exact_round_f32(x: Fraction) -> np.float32:
    """fp32 nearest to the rational x, ties to even, by exhaustive neighbours."""
    f = np.float32(float(x))                   # within one ulp of the answer
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - x),
                                     int(np.array(c, np.float32).view(np.uint32)) & 1))
    return np.float32(best)


def test_round_sum_to_f32_is_a_single_rounding():
    rng = np.random.default_rng(3)
    q = rng.integers(-127, 128, 4000).astype(np.float64)
    s = rng.uniform(1e-3, 1, 4000).astype(np.float32).astype(np.float64)
    ze = (rng.standard_normal(4000) * 10.0 ** rng.integers(-12, 2, 4000)).astype(np.float32).astype(np.float64)
    # crafted double-rounding cases: a = 1 (fp32), b = 2^-24 (1 + 2^-30) straddles a tie
    q = np.concatenate([q, [1.0, 1.0, -1.0]])
    s = np.concatenate([s, [1.0, 1.0, 1.0]])
    ze = np.concatenate([ze, [2.0 ** -24 + 2.0 ** -60, 2.0 ** -24 - 2.0 ** -60, -(2.0 ** -24 + 2.0 ** -60)]])
    got = oracle.round_sum_to_f32(q * s, ze)
    want = np.array([_exact_round_f32(Fraction(a) + Fraction(b)) for a, b in zip(q * s, ze)])
    np.testing.assert_array_equal(got, want)
    assert got[-3] == np.nextafter(np.float32(1), np.float32(2))
    assert got[-2] == np.float32(1)


# ---------------------------------------------------------------------------
# masking, greedy selection, verification
# ---------------------------------------------------------------------------

def test_masked_supertoken_is_never_emitted():
    cfg = Config("t", 0, d=512, d_end=64, vocab=8192, n_sub=4096, subset_kind="perm",
                 sessions=1, rows_per_session=3)
    wl = make_workload(cfg)
    we, wc = wl.w_end_bits.copy(), wl.w_cloud_bits.copy()
    vid = plant_masked_supertoken(we, wc, wl.h_bits, 1, wl.subset)
    Wfull = oracle.decode_bf16(np.concatenate([we, wc], axis=1))
    assert np.argmax(oracle.full_head_logits(wl.h_bits, Wfull)[1]) == vid   # the plant works
    cl = oracle.cloud_call(wl.h_bits, 64, wl.subset, 30.0, w_cloud_bits=wc)
    for mode in ("greedy", "sample"):
        ep = oracle.endpoint_call(cl["q"], cl["scale"], wl.h_bits, 64, wl.subset, we, 1, 3,
                                  drafts=np.array([[vid, vid]]), mode=mode, temperature=5.0,
                                  top_p=1.0, seed=1)
        assert vid not in ep["tokens"] and np.all(np.isin(ep["tokens"], wl.subset))
        assert ep["accept"][0] == 0


def test_greedy_ties_go_to_lowest_id():
    f = np.array([[1, 3, 3, 2], [5, 5, 5, 5]], dtype=np.float32)
    tok, pos, gap = oracle.greedy_select(f, np.array([4, 7, 9, 12]))
    np.testing.assert_array_equal(tok, [7, 4])
    np.testing.assert_array_equal(gap, [0, 0])


@pytest.mark.parametrize("k", [0, 1, 2, 4, 7])
def test_accept_length_exhaustive_patterns(k):
    R = k + 1
    pats = list(range(1 << k))
    n = len(pats)
    rng = np.random.default_rng(k)
    tokens = rng.integers(0, 1000, size=n * R).astype(np.int32)
    drafts = np.empty((n, k), dtype=np.int32)
    want = np.empty(n, dtype=np.int32)
    for s, bits in enumerate(pats):
        lead = 0
        while lead < k and (bits >> lead) & 1:
            lead += 1
        want[s] = lead
        for r in range(k):
            t = tokens[s * R + r]
            drafts[s, r] = t if (bits >> r) & 1 else t + 1000   # + 1000 never equals a token
    got = oracle.accept_lengths(tokens, drafts if k else None, n, R)
    np.testing.assert_array_equal(got, want)


# ---------------------------------------------------------------------------
# sampling (eq. 15 + top-p)
# ---------------------------------------------------------------------------

def _rows(f, m):
    return np.repeat(np.asarray(f, np.float32)[None, :], m, axis=0)


def test_sampling_reduces_to_greedy():
    rng = np.random.default_rng(5)
    f = rng.standard_normal((40, 300)).astype(np.float32)
    S = np.sort(rng.choice(5000, 300, replace=False))
    g, _, gap = oracle.greedy_select(f, S)
    t1, _ = oracle.sample_select(f, S, 1e-4, 1.0, 99, 5)     # tau -> 0
    t2, info = oracle.sample_select(f, S, 0.7, 1e-7, 99, 5)   # top_p -> 0: nucleus = {argmax}
    ok = gap > 1e-2
    np.testing.assert_array_equal(t1[ok], g[ok])
    np.testing.assert_array_equal(t2, g)
    assert np.all(info["nucleus"] == 1)


def test_sampling_chi_square_against_softmax():
    from scipy import stats
    tau = 0.7
    f = np.array([0.3, -0.4, 1.1, 0.0], dtype=np.float32)
    S = np.array([3, 8, 20, 21])
    n = 6000
    tok, _ = oracle.sample_select(_rows(f, n), S, tau, 1.0, 2026, 6)
    p = np.exp(f.astype(np.float64) / np.float32(tau).astype(np.float64))
    p /= p.sum()
    counts = np.array([(tok == i).sum() for i in S])
    assert stats.chisquare(counts, p * n).pvalue > 1e-4


def test_sampling_nucleus_cut_and_renormalisation():
    from scipy import stats
    tau = 1.0
    p = np.array([0.05, 0.5, 0.15, 0.3])
    f = np.log(p).astype(np.float32)
    S = np.array([1, 2, 3, 4])
    n = 6000
    tok, info = oracle.sample_select(_rows(f, n), S, tau, 0.78, 7, 4)
    assert np.all(info["nucleus"] == 2)                       # 0.5 + 0.3 >= 0.78 > 0.5
    assert set(np.unique(tok)) <= {2, 4}
    counts = np.array([(tok == 2).sum(), (tok == 4).sum()])
    assert stats.chisquare(counts, np.array([0.5, 0.3]) / 0.8 * n).pvalue > 1e-4


def test_sampling_walks_in_ascending_id_order():
    # p = (0.1, 0.2, 0.3, 0.4) on ids (10, 20, 30, 40): the inverse CDF in id order
    # maps u in [0, .1) -> 10, [.1, .3) -> 20, [.3, .6) -> 30, [.6, 1) -> 40.
    p = np.array([0.1, 0.2, 0.3, 0.4])
    f = np.log(p).astype(np.float32)
    S = np.array([10, 20, 30, 40])
    m = 64
    tok, _ = oracle.sample_select(_rows(f, m), S, 1.0, 1.0, 31337, 8)
    pe = np.exp(f.astype(np.float64))
    pe /= pe.sum()
    edges = np.cumsum(pe)
    for row in range(m):
        u = oracle.philox_uniform(31337, row % 8, row // 8)
        assert tok[row] == S[int(np.sum(edges <= u))]


def test_sample_candidates_margin_zero_is_the_sample():
    rng = np.random.default_rng(11)
    f = rng.standard_normal((30, 200)).astype(np.float32)
    S = np.sort(rng.choice(4000, 200, replace=False))
    tok, _ = oracle.sample_select(f, S, 0.7, 0.9, 5, 3)
    cand = oracle.sample_candidates(f, S, 0.7, 0.9, 5, 3, 0.0)
    for m in range(30):
        assert list(cand[m]) == [tok[m]]


def test_sample_candidates_cdf_edge():
    # p = (0.1, 0.2, 0.3, 0.4) on ids (10, 20, 30, 40), no cut: interval edges
    # at 0.1, 0.3, 0.6.  A margin past the target's distance to the nearest
    # edge (but short of the next edge) adds the id on the other side of it,
    # one below that distance does not.
    p = np.array([0.1, 0.2, 0.3, 0.4])
    f = np.log(p).astype(np.float32)
    S = np.array([10, 20, 30, 40])
    pe = np.exp(f.astype(np.float64))
    pe /= pe.sum()
    edges = np.cumsum(pe)[:-1]
    for row in range(24):
        u = oracle.philox_uniform(77, row % 4, row // 4)
        i = int(np.sum(edges <= u))
        dist = np.abs(edges - u)
        k = int(np.argmin(dist))
        other = S[k + 1] if u < edges[k] else S[k]
        d, d2 = np.sort(dist)[:2]
        if not d2 > d:
            continue
        # margins below the nearest edge, and between the nearest and the next
        one = oracle.sample_candidates(_rows(f, 1), S, 1.0, 1.0, 77, 4, d * 0.5, row_index=[row])[0]
        two = oracle.sample_candidates(_rows(f, 1), S, 1.0, 1.0, 77, 4, (d + d2) / 2,
                                       row_index=[row])[0]
        assert list(one) == [S[i]]
        assert sorted(two) == sorted({int(S[i]), int(other)})


def test_sample_candidates_nucleus_cut():
    # p = (0.05, 0.5, 0.15, 0.3) on ids (1, 2, 3, 4), top_p 0.78: the exact
    # nucleus is {2, 4} (0.5 + 0.3 >= 0.78); a margin of 0.025 lets the cut
    # take {2, 3, 4} too (0.95 >= 0.805).  Counted by hand for u in
    # [0.62, 0.64]: nucleus {2, 4} (run 0.5, 0.8) puts the target 0.8u in
    # [0.496, 0.512], within 0.025 of the edge 0.5 -> ids 2 and 4; nucleus
    # {2, 3, 4} (run 0.5, 0.65, 0.95) puts 0.95u in [0.589, 0.608], whose
    # window [0.564, 0.633] lies inside id 3's interval [0.5, 0.65) -> id 3.
    p = np.array([0.05, 0.5, 0.15, 0.3])
    f = np.log(p).astype(np.float32)
    S = np.array([1, 2, 3, 4])
    hits = 0
    for row in range(4000):
        u = oracle.philox_uniform(9, row % 4, row // 4)
        if not (0.62 <= u <= 0.64):
            continue
        c = oracle.sample_candidates(_rows(f, 1), S, 1.0, 0.78, 9, 4, 0.025, row_index=[row])[0]
        assert list(c) == [2, 3, 4]
        c0 = oracle.sample_candidates(_rows(f, 1), S, 1.0, 0.78, 9, 4, 0.0, row_index=[row])[0]
        assert list(c0) == [2 if 0.8 * u < 0.5 else 4]
        hits += 1
    assert hits >= 20


def test_philox_uniform_takes_the_top_24_bits_of_word_0():
    # seed 0, row 0, session 0 is counter 0 / key 0: word 0 of the first known answer
    assert oracle.philox_uniform(0, 0, 0) == (0x6627E8D5 >> 8) * 2.0 ** -24
    # seed = all ones is key (0xffffffff, 0xffffffff); counter (row, session, 0, 0)
    x0 = oracle.philox4x32_10((3, 5, 0, 0), (0xFFFFFFFF, 0xFFFFFFFF))[0]
    assert oracle.philox_uniform(2 ** 64 - 1, 3, 5) == (x0 >> 8) * 2.0 ** -24
