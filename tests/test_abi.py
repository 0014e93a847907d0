"""The C-ABI library: it loads, exports what include/*.h declare, and its
host-side validation rejects bad arguments before touching any device."""

import ctypes
import glob
import os
import re

import numpy as np
import pytest

from paper_2607_13093_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for path in sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))):
        text = re.sub(r"/\*.*?\*/", "", open(path).read(), flags=re.S)
        names |= set(re.findall(r"\b(sph_[a-z_]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert len(names) >= 10
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(_lib.SIGNATURES), "binding signatures out of sync with include/*.h"


def test_abi_version(lib):
    assert lib.sph_abi_version() == 1
    assert lib.sph_last_error() == b""


def test_debug_sync_switch(lib):
    # a query leaves the state alone; each switch returns the previous state
    start = lib.sph_debug_sync(-1)
    assert start in (0, 1)
    assert lib.sph_debug_sync(1) == start
    assert lib.sph_debug_sync(-1) == 1
    assert lib.sph_debug_sync(0) == 1
    assert lib.sph_debug_sync(-1) == 0
    lib.sph_debug_sync(start)


def _create(lib, ids, vocab):
    arr = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
    out = ctypes.c_void_p(123)
    rc = lib.sph_subset_create(arr.ctypes.data if arr.size else None, arr.size, vocab, None, out)
    return rc, out


@pytest.mark.parametrize("ids,vocab,code,msg", [
    ([3, 2, 5], 10, _lib.SPH_E_SUBSET, "ascending"),
    ([1, 1, 2], 10, _lib.SPH_E_SUBSET, "ascending"),
    ([0, 4, 10], 10, _lib.SPH_E_SUBSET, "outside"),
    ([-1, 4], 10, _lib.SPH_E_SUBSET, "outside"),
    (list(range(11)), 10, _lib.SPH_E_SUBSET, "size"),
    ([1, 2], 0, _lib.SPH_E_INVALID_ARG, "vocab"),
])
def test_subset_validation(lib, ids, vocab, code, msg):
    rc, out = _create(lib, ids, vocab)
    assert rc == code
    assert msg in lib.sph_last_error().decode()
    assert out.value is None  # nothing created


def test_subset_empty_and_null(lib):
    out = ctypes.c_void_p()
    one = np.zeros(1, np.int32)
    assert lib.sph_subset_create(one.ctypes.data, 0, 10, None, out) == _lib.SPH_E_SUBSET
    assert lib.sph_subset_create(None, 3, 10, None, out) == _lib.SPH_E_INVALID_ARG
    assert lib.sph_subset_create(one.ctypes.data, 1, 10, None, None) == _lib.SPH_E_INVALID_ARG
    assert lib.sph_subset_create_full(0, None, out) == _lib.SPH_E_INVALID_ARG
    assert lib.sph_subset_size(None, None, None) == _lib.SPH_E_INVALID_ARG
    lib.sph_subset_destroy(None)
    assert lib.sph_cloud_partial_workspace(5, None) == 0
    assert lib.sph_fuse_verify_workspace(5, None, 0) == 0


def _cloud(lib, **kw):
    a = dict(h=1, ldh=64, M=3, d=64, w=16, ldw=64, wtype=_lib.SPH_W_BF16, ws_scale=None,
             bias=None, subset=None, clip=30.0, q=1, s=1, z=None, work=1, nbytes=0)
    a.update(kw)
    return lib.sph_cloud_partial(a["h"], a["ldh"], a["M"], a["d"], a["w"], a["ldw"], a["wtype"],
                                 a["ws_scale"], a["bias"], a["subset"], a["clip"], a["q"], a["s"],
                                 a["z"], a["work"], a["nbytes"], None)


@pytest.mark.parametrize("kw,msg", [
    (dict(M=-1), "M=-1"),
    (dict(d=-4), "d_cloud"),
    (dict(wtype=7), "weight type"),
    (dict(wtype=_lib.SPH_W_FP8_E4M3), "w_row_scale"),
    (dict(ws_scale=64), "only for fp8"),
    (dict(clip=0.0), "clip_c"),
    (dict(clip=float("inf")), "clip_c"),
    (dict(clip=float("nan")), "clip_c"),
    (dict(ldh=32), "row strides"),
    (dict(ldw=32), "row strides"),
    (dict(), "subset is NULL"),
])
def test_cloud_partial_validation(lib, kw, msg):
    assert _cloud(lib, **kw) == _lib.SPH_E_INVALID_ARG
    assert msg in lib.sph_last_error().decode()


def _fuse(lib, **kw):
    a = dict(q=1, s=1, h=1, ldh=64, d=64, w=16, ldw=64, subset=None, S=2, R=3, drafts=1,
             mode=_lib.SPH_GREEDY, temp=1.0, top_p=1.0, seed=0, tok=1, acc=1, f=None,
             work=1, nbytes=0)
    a.update(kw)
    return lib.sph_fuse_verify(a["q"], a["s"], a["h"], a["ldh"], a["d"], a["w"], a["ldw"],
                               a["subset"], a["S"], a["R"], a["drafts"], a["mode"], a["temp"],
                               a["top_p"], a["seed"], a["tok"], a["acc"], a["f"], a["work"],
                               a["nbytes"], None)


@pytest.mark.parametrize("kw,msg", [
    (dict(S=-1), "n_sessions"),
    (dict(R=0), "rows_per_session"),
    (dict(R=5000), "rows_per_session"),
    (dict(d=-1), "d_end"),
    (dict(mode=9), "mode"),
    (dict(mode=_lib.SPH_SAMPLE, temp=0.0), "temperature"),
    (dict(mode=_lib.SPH_SAMPLE, temp=float("nan")), "temperature"),
    (dict(mode=_lib.SPH_SAMPLE, top_p=0.0), "top_p"),
    (dict(mode=_lib.SPH_SAMPLE, top_p=1.5), "top_p"),
    (dict(ldh=16), "row strides"),
    (dict(), "subset is NULL"),
])
def test_fuse_verify_validation(lib, kw, msg):
    assert _fuse(lib, **kw) == _lib.SPH_E_INVALID_ARG
    assert msg in lib.sph_last_error().decode()


@pytest.mark.parametrize("bits,block,msg", [
    (2, 0, "bits=2"),
    (16, 0, "bits=16"),
    (8, 128, "block=128"),
    (4, 300, "block=300"),
    (4, 8192, "block=8192"),
    (8, -256, "block=-256"),
])
def test_payload_format_validation(lib, bits, block, msg):
    # both halves reject a payload format they do not implement, before any
    # other argument is looked at
    rc = lib.sph_cloud_partial_fmt(1, 64, 3, 64, 16, 64, _lib.SPH_W_BF16, None, None, None, 30.0,
                                   bits, block, 1, 1, None, 1, 0, None)
    assert rc == _lib.SPH_E_INVALID_ARG
    assert msg in lib.sph_last_error().decode()
    rc = lib.sph_fuse_verify_fmt(1, 1, bits, block, 1, 64, 64, 16, 64, None, 2, 3, 1,
                                 _lib.SPH_GREEDY, 1.0, 1.0, 0, 1, 1, None, 1, 0, None)
    assert rc == _lib.SPH_E_INVALID_ARG
    assert msg in lib.sph_last_error().decode()


@pytest.mark.parametrize("n,bits,block,code_bytes,scales", [
    (0, 8, 0, 0, 1),
    (1, 4, 256, 1, 1),
    (5, 4, 0, 3, 1),
    (49153, 8, 0, 49153, 1),
    (49153, 4, 1024, 24577, 49),
    (4096, 4, 4096, 2048, 1),
    (4097, 8, 4096, 4097, 2),
])
def test_payload_sizes(lib, n, bits, block, code_bytes, scales):
    # eq. 21: ceil(n * b / 8) code bytes plus the scales of the row
    assert lib.sph_payload_code_bytes(n, bits) == code_bytes
    assert lib.sph_payload_scale_count(n, block) == scales


def test_payload_sizes_reject(lib):
    assert lib.sph_payload_code_bytes(5, 3) == -1
    assert lib.sph_payload_code_bytes(-1, 8) == -1
    assert lib.sph_payload_scale_count(5, 300) == -1
    assert lib.sph_payload_scale_count(-5, 0) == -1


@pytest.mark.parametrize("kw,msg", [
    (dict(M=-1), "M=-1"),
    (dict(d=-3), "d=-3"),
    (dict(ldh=100), "row strides"),
    (dict(ldq=100), "row strides"),
    (dict(h=None), "NULL"),
    (dict(q=None), "NULL"),
    (dict(s=None), "NULL"),
])
def test_hidden_quantize_validation(lib, kw, msg):
    a = dict(h=16, ldh=256, M=3, d=256, q=16, ldq=256, s=16)
    a.update(kw)
    rc = lib.sph_hidden_quantize(a["h"], a["ldh"], a["M"], a["d"], a["q"], a["ldq"], a["s"], None)
    assert rc == _lib.SPH_E_INVALID_ARG
    assert msg in lib.sph_last_error().decode()


def test_hidden_quantize_empty_batch_launches_nothing(lib):
    assert lib.sph_hidden_quantize(None, 8, 0, 8, None, 8, None, None) == 0


def test_fuse_verify_hq_validation(lib):
    # strides are checked before anything else needs the subset or a device
    rc = lib.sph_fuse_verify_hq(1, 1, 8, 0, 1, 32, 1, 64, 16, 64, None, 2, 3, 1,
                                _lib.SPH_GREEDY, 1.0, 1.0, 0, 1, 1, None, 1, 0, None)
    assert rc == _lib.SPH_E_INVALID_ARG
    assert "row strides" in lib.sph_last_error().decode()
    rc = lib.sph_fuse_verify_hq(1, 1, 5, 0, 1, 64, 1, 64, 16, 64, None, 2, 3, 1,
                                _lib.SPH_GREEDY, 1.0, 1.0, 0, 1, 1, None, 1, 0, None)
    assert rc == _lib.SPH_E_INVALID_ARG and b"bits=5" in lib.sph_last_error()
    assert lib.sph_fuse_verify_hq_workspace(5, 256, None, 0) == 0


def test_gcm_validation(lib):
    # rejected on the host before any device access
    E = _lib.SPH_E_INVALID_ARG
    assert lib.sph_gcm_seal(None, 1, 16, 1, 16, 1, None, 0, 0, 1, 16, 1, 1, 1 << 20, None) == E
    assert b"key is NULL" in lib.sph_last_error()
    out = ctypes.c_void_p()
    key = (ctypes.c_uint8 * 24)()
    assert lib.sph_gcm_key_create(key, 24, None, out) == E and b"key_bytes=24" in lib.sph_last_error()
    assert lib.sph_gcm_key_create(None, 16, None, out) == E
    assert lib.sph_gcm_key_create(key, 16, None, None) == E
    lib.sph_gcm_key_destroy(None)


def _segs(*specs):
    arr = (_lib.GcmSegment * max(len(specs), 1))()
    for k, (src, ld_in, dst, ld_out, nb) in enumerate(specs):
        arr[k] = _lib.GcmSegment(src, ld_in, dst, ld_out, nb)
    return arr


@pytest.mark.parametrize("segs,nseg,rows,aad,code,msg", [
    (_segs((1, 16, 1, 16, 16)), 0, 1, 0, -1, b"nseg=0"),
    (_segs(*[(1, 16, 1, 16, 16)] * 4), 5, 1, 0, -1, b"nseg=5"),
    (None, 1, 1, 0, -1, b"segments NULL"),
    (_segs((1, 16, 1, 16, 16), (1, 8, 1, 8, -1)), 2, 1, 0, -1, b"segment 1 has -1 bytes"),
    (_segs((1, 16, 1, 16, 16), (1, 7, 1, 8, 8)), 2, 1, 0, -1, b"segment 1: row strides"),
    (_segs((1, 16, 1, 16, 16), (None, 8, 1, 8, 8)), 2, 1, 0, -1, b"segment 1: input/output is NULL"),
    (_segs((1, 16, 1, 16, 16), (1, 8, 1, 8, 8)), 2, 65536, 0, -1, b"rows=65536"),
    (_segs((1, 1 << 18, 1, 1 << 18, 1 << 17), (1, 1 << 18, 1, 1 << 18, 1 << 17)), 2, 1, 0, -3,
     b"exceeds 16384 blocks"),
    (_segs((1, 16, 1, 16, 16)), 1, 1, 2000, -1, b"aad_bytes=2000"),
])
def test_gcm_segment_validation(lib, segs, nseg, rows, aad, code, msg):
    # a dummy key handle: every case is rejected on the host before the key
    # or any buffer is touched
    rc = lib.sph_gcm_seal_segments(1, segs, nseg, rows, 1, 1, 2048, aad, 1, 1, 1 << 20, None)
    assert rc == code and msg in lib.sph_last_error(), lib.sph_last_error()
    rc = lib.sph_gcm_open_segments(1, segs, nseg, rows, 1, 1, 2048, aad, 1, 1, 1, 1 << 20, None)
    assert rc == code and msg in lib.sph_last_error(), lib.sph_last_error()


def test_gcm_segments_empty_batch_and_empty_segment(lib):
    # zero rows, and an empty segment with NULL pointers, launch nothing
    segs = _segs((None, 0, None, 0, 0), (1, 16, 1, 16, 16))
    assert lib.sph_gcm_seal_segments(1, segs, 2, 0, None, None, 0, 0, None, None, 0, None) == 0
    assert lib.sph_gcm_workspace(0, 16) == 0


@pytest.mark.parametrize("rows,row_bytes,need", [
    (0, 100, 0), (5, 0, 256), (1, 1, 256), (5, 49152, 1280), (2048, 32768, 2048 * 16),
    (3, 16 * 256 + 1, 256), (16, 16 * 256, 512), (16, 16 * 257, 512), (40, 52429, 2048),
    (64, 123457, 64 * 2 * 16),
])
def test_gcm_workspace_sizes(lib, rows, row_bytes, need):
    # one 16-byte partial sum per row and workgroup of 256 threads, each
    # thread chaining k = clamp(ceil(rows * blocks / 32768), 1, 16) blocks;
    # for k = 1 one more workgroup when the last has fewer than 66 threads
    # without a block (room for the largest AAD); rounded up to 256 bytes
    assert lib.sph_gcm_workspace(rows, row_bytes) == need


def test_error_string_is_thread_local(lib):
    import threading
    assert _cloud(lib, M=-1) == _lib.SPH_E_INVALID_ARG
    seen = {}

    def other():
        seen["msg"] = lib.sph_last_error()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen["msg"] == b""
    assert b"M=-1" in lib.sph_last_error()


@pytest.mark.parametrize("buf,nbytes,sink,msg", [
    (0, 1024, 64, "NULL"),
    (16, 1024, 0, "NULL"),
    (24, 1024, 64, "16-byte aligned"),
    (16, 1000, 64, "multiple of 16"),
    (16, 0, 64, "multiple of 16"),
])
def test_probe_read_validation(lib, buf, nbytes, sink, msg):
    # rejected on the host: no pointer is dereferenced, nothing is launched
    assert lib.sph_probe_read(buf, nbytes, sink, None) == _lib.SPH_E_INVALID_ARG
    assert msg in lib.sph_last_error().decode()


@pytest.mark.parametrize("iters,sink,with_out,msg", [
    (0, 64, True, "iters"),
    ((1 << 30) + 1, 64, True, "iters"),
    (10, 0, True, "NULL"),
    (10, 64, False, "NULL"),
])
def test_probe_mfma_validation(lib, iters, sink, with_out, msg):
    flops = ctypes.c_double(0.0)
    out = ctypes.byref(flops) if with_out else None
    assert lib.sph_probe_mfma(iters, sink, None, out) == _lib.SPH_E_INVALID_ARG
    assert msg in lib.sph_last_error().decode()
