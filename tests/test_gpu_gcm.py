"""GPU parity of the AES-GCM payload seal (eq. 19) against the CPU oracle
(oracle/gcm.py): ciphertexts and tags bit for bit, authenticated opening,
tamper detection per row, in-place operation, strided rows, messages made
of several row segments (codes and scales as one message), and a payload
sealed between the two halves of the projection."""

import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import gcm as ogcm
import paper_2607_13093_amd as sph
from synth import CONFIGS, Config, make_workload

import parity as P

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


CASES = [
    # (key bytes, rows, row bytes, aad bytes)
    (16, 1, 0, 0),
    (16, 3, 1, 5),
    (16, 2, 15, 16),
    (32, 4, 16, 0),
    (16, 5, 17, 40),
    (32, 3, 4099, 13),
    (16, 33, 300, 24),
    (16, 5, 49152, 24),     # the decode payload's code rows
    (32, 2, 65536, 1024),   # 4096 + 64 + 1 blocks, the largest AAD
]


@pytest.mark.parametrize("case", CASES, ids=[f"k{k}r{r}L{l}a{a}" for k, r, l, a in CASES])
def test_seal_matches_oracle_and_opens(case):
    klen, rows, L, la = case
    rng = np.random.default_rng(7 * rows + L + la + klen)
    key = rng.bytes(klen)
    pt = rng.integers(0, 256, (rows, L), dtype=np.uint8)
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    aad = rng.integers(0, 256, (rows, la), dtype=np.uint8)
    ct_ref, tag_ref = ogcm.seal_rows(key, pt, iv, aad)
    say(f"[gpu] gcm seal key={klen} rows={rows} L={L} aad={la}")
    k = sph.GcmKey(key)
    ct, tag = sph.gcm_seal(k, _dev(pt), _dev(iv), _dev(aad) if la else None)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(ct), ct_ref)
    np.testing.assert_array_equal(P.host(tag), tag_ref)
    say(f"[gpu] gcm open key={klen} rows={rows} L={L}")
    back, ok = sph.gcm_open(k, ct, _dev(iv), tag, _dev(aad) if la else None)
    torch.cuda.synchronize()
    assert P.host(ok).tolist() == [1] * rows
    np.testing.assert_array_equal(P.host(back), pt)


def test_large_batch():
    # 40 rows x 3277 blocks (2 MB, ragged last block, AAD): the size of a
    # batched payload; three rows checked against the oracle
    rng = np.random.default_rng(31)
    key = rng.bytes(32)
    rows, L, la = 40, 52429, 24
    pt = rng.integers(0, 256, (rows, L), dtype=np.uint8)
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    aad = rng.integers(0, 256, (rows, la), dtype=np.uint8)
    say(f"[gpu] gcm chunked rows={rows} L={L}")
    k = sph.GcmKey(key)
    ct, tag = sph.gcm_seal(k, _dev(pt), _dev(iv), _dev(aad))
    torch.cuda.synchronize()
    ct_h, tag_h = P.host(ct), P.host(tag)
    check = [0, 17, 39]                      # the oracle is slow: three rows
    ct_ref, tag_ref = ogcm.seal_rows(key, pt[check], iv[check], aad[check])
    np.testing.assert_array_equal(ct_h[check], ct_ref)
    np.testing.assert_array_equal(tag_h[check], tag_ref)
    bad = ct_h.copy()
    bad[5, 30000] ^= 0x04
    back, ok = sph.gcm_open(k, _dev(bad), _dev(iv), _dev(tag_h), _dev(aad))
    torch.cuda.synchronize()
    okh = P.host(ok)
    assert okh[5] == 0 and okh.sum() == rows - 1
    np.testing.assert_array_equal(np.delete(P.host(back), 5, axis=0), np.delete(pt, 5, axis=0))


def test_longest_chains_with_a_ragged_part():
    # 64 rows x 7717 blocks: every thread chains 16 blocks (two workgroups
    # per row, the second ragged); two rows checked against the oracle, all
    # rows opened, one tampered row rejected
    rng = np.random.default_rng(33)
    key = rng.bytes(16)
    rows, L, la = 64, 123457, 13
    pt = rng.integers(0, 256, (rows, L), dtype=np.uint8)
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    aad = rng.integers(0, 256, (rows, la), dtype=np.uint8)
    say(f"[gpu] gcm chained rows={rows} L={L}")
    k = sph.GcmKey(key)
    ct, tag = sph.gcm_seal(k, _dev(pt), _dev(iv), _dev(aad))
    torch.cuda.synchronize()
    ct_h, tag_h = P.host(ct), P.host(tag)
    for m in (0, rows - 1):
        c, t = ogcm.gcm_encrypt(key, iv[m].tobytes(), pt[m].tobytes(), aad[m].tobytes())
        assert ct_h[m].tobytes() == c and tag_h[m].tobytes() == t
    ct_h = ct_h.copy()
    ct_h[17, L - 1] ^= 4
    back, ok = sph.gcm_open(k, _dev(ct_h), _dev(iv), tag, _dev(aad))
    torch.cuda.synchronize()
    okh = P.host(ok)
    assert okh[17] == 0 and okh.sum() == rows - 1
    np.testing.assert_array_equal(np.delete(P.host(back), 17, axis=0), np.delete(pt, 17, axis=0))


def test_open_flags_exactly_the_tampered_rows():
    rng = np.random.default_rng(21)
    key = rng.bytes(16)
    rows, L, la = 6, 1000, 20
    pt = rng.integers(0, 256, (rows, L), dtype=np.uint8)
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    aad = rng.integers(0, 256, (rows, la), dtype=np.uint8)
    k = sph.GcmKey(key)
    say("[gpu] gcm tamper")
    ct, tag = sph.gcm_seal(k, _dev(pt), _dev(iv), _dev(aad))
    ct_h, tag_h, aad_t, iv_t = P.host(ct).copy(), P.host(tag).copy(), aad.copy(), iv.copy()
    ct_h[1, 999] ^= 0x01        # last ciphertext byte
    tag_h[2, 0] ^= 0x80         # tag
    aad_t[3, 7] ^= 0x10         # associated data
    iv_t[4, 11] ^= 0x01         # nonce
    ct_h[5, 0] ^= 0x00          # untouched
    back, ok = sph.gcm_open(k, _dev(ct_h), _dev(iv_t), _dev(tag_h), _dev(aad_t))
    torch.cuda.synchronize()
    assert P.host(ok).tolist() == [1, 0, 0, 0, 0, 1]
    np.testing.assert_array_equal(P.host(back)[[0, 5]], pt[[0, 5]])


def test_in_place_and_strided_rows():
    rng = np.random.default_rng(22)
    key = rng.bytes(32)
    rows, L, ld = 4, 777, 1024
    buf = rng.integers(0, 256, (rows, ld), dtype=np.uint8)
    pt = buf[:, :L].copy()
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    ct_ref, tag_ref = ogcm.seal_rows(key, pt, iv, np.zeros((rows, 0), np.uint8))
    k = sph.GcmKey(key)
    say("[gpu] gcm in place, strided")
    d = _dev(buf)
    view = d[:, :L]
    tag = torch.empty((rows, 16), dtype=torch.uint8, device="cuda")
    sph.gcm_seal(k, view, _dev(iv), None, out=(view, tag))
    torch.cuda.synchronize()
    got = P.host(d)
    np.testing.assert_array_equal(got[:, :L], ct_ref)
    np.testing.assert_array_equal(got[:, L:], buf[:, L:])          # bytes past each row untouched
    np.testing.assert_array_equal(P.host(tag), tag_ref)
    ok = torch.empty((rows,), dtype=torch.int32, device="cuda")
    sph.gcm_open(k, view, _dev(iv), tag, None, out=(view, ok))
    torch.cuda.synchronize()
    assert P.host(ok).tolist() == [1] * rows
    np.testing.assert_array_equal(P.host(d)[:, :L], pt)


def test_sealed_payload_between_the_halves():
    # cloud partial -> seal codes and scales -> open -> endpoint call; the
    # endpoint's results equal those on the unsealed payload bit for bit
    cfg = Config("gcm_payload", 95, d=1032, d_end=64, vocab=6000, n_sub=2501, subset_kind="choice",
                 sessions=3, rows_per_session=4)
    wl = make_workload(cfg)
    dw = P.DeviceWorkload(wl)
    say("[gpu] gcm sealed payload, b=4 block=256")
    q, s, _ = dw.cloud(want_z=False, bits=4, block=256)
    rng = np.random.default_rng(23)
    key = rng.bytes(16)
    k = sph.GcmKey(key)
    M = cfg.M
    # nonces: (session, message type, row) -- distinct for every message
    iv = np.zeros((2, M, 12), np.uint8)
    for t in range(2):
        for m in range(M):
            iv[t, m, :4] = np.frombuffer(np.uint32(m // cfg.rows_per_session).tobytes()[::-1], np.uint8)
            iv[t, m, 4] = t
            iv[t, m, 8:] = np.frombuffer(np.uint32(m).tobytes()[::-1], np.uint8)
    aad = np.tile(np.frombuffer(b"session-meta", np.uint8), (M, 1))
    cq, tq = sph.gcm_seal(k, q, _dev(iv[0]), _dev(aad))
    cs, ts = sph.gcm_seal(k, s.view(torch.uint8).reshape(M, -1), _dev(iv[1]), _dev(aad))
    torch.cuda.synchronize()
    ct_ref, tag_ref = ogcm.seal_rows(key, P.host(q).view(np.uint8), iv[0], aad)
    np.testing.assert_array_equal(P.host(cq), ct_ref)
    np.testing.assert_array_equal(P.host(tq), tag_ref)
    q2, okq = sph.gcm_open(k, cq, _dev(iv[0]), tq, _dev(aad))
    s2, oks = sph.gcm_open(k, cs, _dev(iv[1]), ts, _dev(aad))
    torch.cuda.synchronize()
    assert P.host(okq).all() and P.host(oks).all()
    s2 = s2.view(torch.float32).reshape(s.shape)
    drafts = np.zeros((cfg.sessions, cfg.k), np.int32)
    t1, a1, f1 = dw.fuse(q, s, drafts, bits=4, block=256)
    t2, a2, f2 = dw.fuse(q2, s2, drafts, bits=4, block=256)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(q2), P.host(q))
    np.testing.assert_array_equal(P.host(t2), P.host(t1))
    np.testing.assert_array_equal(P.host(f2).view(np.uint32), P.host(f1).view(np.uint32))


SEG_CASES = [
    # (key bytes, rows, segment lengths, aad bytes)
    (16, 3, (40, 12), 24),             # codes + scales of a small payload row
    (16, 5, (0, 17, 0, 33), 5),        # empty segments around ragged ones
    (32, 4, (5, 16, 1, 33), 0),        # boundaries inside, at and across blocks
    (16, 2, (49152, 4), 24),           # decode payload row, 8 bits: codes, then the row scale
    (16, 5, (24576, 768), 24),         # 4 bits, block 256: codes, then 192 block scales
    (32, 7, (1, 1, 1, 1), 16),
    (16, 3, (16 * 300, 16 * 300 + 3), 1024),
]


@pytest.mark.parametrize("case", SEG_CASES, ids=[f"k{k}r{r}s{'-'.join(map(str, s))}a{a}"
                                                 for k, r, s, a in SEG_CASES])
def test_segments_seal_the_concatenated_rows(case):
    # one message per row = row m of every segment in order; the segments
    # live in separate strided buffers with bytes between their rows
    klen, rows, lens, la = case
    rng = np.random.default_rng(sum(lens) + 13 * rows + la + klen)
    key = rng.bytes(klen)
    parts = [rng.integers(0, 256, (rows, n), dtype=np.uint8) for n in lens]
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    aad = rng.integers(0, 256, (rows, la), dtype=np.uint8)
    msg = np.concatenate(parts, axis=1)
    ct_ref, tag_ref = ogcm.seal_rows(key, msg, iv, aad)
    pad_in = [rng.integers(0, 256, (rows, n + 7), dtype=np.uint8) for n in lens]
    for p, q in zip(pad_in, parts):
        p[:, :q.shape[1]] = q
    bufs = [_dev(p) for p in pad_in]
    ins = [b[:, :n] for b, n in zip(bufs, lens)]
    outs_buf = [torch.full((rows, n + 9), 0xA5, dtype=torch.uint8, device="cuda") for n in lens]
    outs = [b[:, :n] for b, n in zip(outs_buf, lens)]
    say(f"[gpu] gcm segments seal key={klen} rows={rows} segs={lens} aad={la}")
    k = sph.GcmKey(key)
    cts, tag = sph.gcm_seal_segments(k, ins, _dev(iv), _dev(aad) if la else None, out=outs)
    torch.cuda.synchronize()
    got = np.concatenate([P.host(c) for c in cts], axis=1) if sum(lens) else np.zeros((rows, 0), np.uint8)
    np.testing.assert_array_equal(got, ct_ref)
    np.testing.assert_array_equal(P.host(tag), tag_ref)
    for b, n in zip(outs_buf, lens):
        assert (P.host(b)[:, n:] == 0xA5).all()                      # bytes past each row untouched
    say(f"[gpu] gcm segments open key={klen} rows={rows} segs={lens}")
    back, ok = sph.gcm_open_segments(k, cts, _dev(iv), tag, _dev(aad) if la else None)
    torch.cuda.synchronize()
    assert P.host(ok).tolist() == [1] * rows
    for b, p in zip(back, parts):
        np.testing.assert_array_equal(P.host(b), p)
    # the same messages sealed as one contiguous batch agree
    ct1, tag1 = sph.gcm_seal(k, _dev(msg), _dev(iv), _dev(aad) if la else None)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(ct1), ct_ref)
    np.testing.assert_array_equal(P.host(tag1), tag_ref)


def test_segments_in_place_and_tamper():
    rng = np.random.default_rng(24)
    key = rng.bytes(16)
    rows, lens = 5, (100, 36, 7)
    parts = [rng.integers(0, 256, (rows, n), dtype=np.uint8) for n in lens]
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    ct_ref, tag_ref = ogcm.seal_rows(key, np.concatenate(parts, axis=1), iv,
                                     np.zeros((rows, 0), np.uint8))
    k = sph.GcmKey(key)
    say("[gpu] gcm segments in place")
    d = [_dev(p) for p in parts]
    _, tag = sph.gcm_seal_segments(k, d, _dev(iv), None, out=d)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(np.concatenate([P.host(x) for x in d], axis=1), ct_ref)
    np.testing.assert_array_equal(P.host(tag), tag_ref)
    # a flipped byte in any segment fails exactly its own row
    d[0][1, 99] ^= 1
    d[1][3, 0] ^= 0x40
    d[2][4, 6] ^= 0x02
    say("[gpu] gcm segments open, tampered rows 1, 3, 4")
    _, ok = sph.gcm_open_segments(k, d, _dev(iv), tag, None, out=d)
    torch.cuda.synchronize()
    assert P.host(ok).tolist() == [1, 0, 1, 0, 0]
    for x, p in zip(d, parts):
        np.testing.assert_array_equal(P.host(x)[[0, 2]], p[[0, 2]])


def test_segments_seal_a_payload_as_one_message():
    # cloud partial -> one message per row (codes, then the row's block
    # scales) -> open -> endpoint call, identical to the unsealed payload
    cfg = Config("gcm_segments", 96, d=1032, d_end=64, vocab=6000, n_sub=2501, subset_kind="choice",
                 sessions=3, rows_per_session=4)
    wl = make_workload(cfg)
    dw = P.DeviceWorkload(wl)
    say("[gpu] gcm payload as one message, b=4 block=256")
    q, s, _ = dw.cloud(want_z=False, bits=4, block=256)
    rng = np.random.default_rng(25)
    key = rng.bytes(16)
    k = sph.GcmKey(key)
    M = cfg.M
    iv = rng.integers(0, 256, (M, 12), dtype=np.uint8)
    aad = np.tile(np.frombuffer(b"session-meta", np.uint8), (M, 1))
    s_bytes = s.view(torch.uint8).reshape(M, -1)
    (cq, cs), tag = sph.gcm_seal_segments(k, [q, s_bytes], _dev(iv), _dev(aad))
    torch.cuda.synchronize()
    msg = np.concatenate([P.host(q).view(np.uint8).reshape(M, -1), P.host(s_bytes)], axis=1)
    ct_ref, tag_ref = ogcm.seal_rows(key, msg, iv, aad)
    np.testing.assert_array_equal(np.concatenate([P.host(cq), P.host(cs)], axis=1), ct_ref)
    np.testing.assert_array_equal(P.host(tag), tag_ref)
    (q2, s2), ok = sph.gcm_open_segments(k, [cq, cs], _dev(iv), tag, _dev(aad))
    torch.cuda.synchronize()
    assert P.host(ok).all()
    q2 = q2.view(q.dtype).reshape(q.shape)
    s2 = s2.view(torch.float32).reshape(s.shape)
    drafts = np.zeros((cfg.sessions, cfg.k), np.int32)
    t1, a1, f1 = dw.fuse(q, s, drafts, bits=4, block=256)
    t2, a2, f2 = dw.fuse(q2, s2, drafts, bits=4, block=256)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(P.host(t2), P.host(t1))
    np.testing.assert_array_equal(P.host(a2), P.host(a1))
    np.testing.assert_array_equal(P.host(f2).view(np.uint32), P.host(f1).view(np.uint32))


def test_limits_most_rows_and_longest_message():
    # 65535 one-byte messages (the largest grid), six checked against the
    # oracle and all opened; then one message of the largest length (16383
    # data blocks + the length block, no AAD) and one byte more, refused
    rng = np.random.default_rng(41)
    key = rng.bytes(16)
    rows = 65535
    pt = rng.integers(0, 256, (rows, 1), dtype=np.uint8)
    iv = rng.integers(0, 256, (rows, 12), dtype=np.uint8)
    say(f"[gpu] gcm rows={rows} L=1")
    k = sph.GcmKey(key)
    ct, tag = sph.gcm_seal(k, _dev(pt), _dev(iv))
    torch.cuda.synchronize()
    ct_h, tag_h = P.host(ct), P.host(tag)
    for m in (0, 1, 255, 256, 40000, rows - 1):
        c, t = ogcm.gcm_encrypt(key, iv[m].tobytes(), pt[m].tobytes())
        assert ct_h[m].tobytes() == c and tag_h[m].tobytes() == t
    back, ok = sph.gcm_open(k, ct, _dev(iv), tag)
    torch.cuda.synchronize()
    assert int(P.host(ok).sum()) == rows
    np.testing.assert_array_equal(P.host(back), pt)

    L = 16 * 16383
    pt1 = rng.integers(0, 256, (1, L), dtype=np.uint8)
    iv1 = rng.integers(0, 256, (1, 12), dtype=np.uint8)
    say(f"[gpu] gcm rows=1 L={L}")
    ct1, tag1 = sph.gcm_seal(k, _dev(pt1), _dev(iv1))
    torch.cuda.synchronize()
    c, t = ogcm.gcm_encrypt(key, iv1[0].tobytes(), pt1[0].tobytes())
    assert P.host(ct1)[0].tobytes() == c and P.host(tag1)[0].tobytes() == t
    with pytest.raises(sph.SphError, match="exceeds 16384 blocks"):
        sph.gcm_seal(k, _dev(np.zeros((1, L + 1), np.uint8)), _dev(iv1))
