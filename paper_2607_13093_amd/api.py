"""Thin torch-facing binding of libsph: argument marshalling only.

torch supplies device memory and the current stream; every step of the
computation runs in the library's HIP kernels.  Tensors must live on the GPU
and be contiguous along their last dimension (row strides are passed on).
"""

from __future__ import annotations

from typing import Optional

import torch

from . import _lib
from ._lib import SphError, check  # noqa: F401

GREEDY = _lib.SPH_GREEDY
SAMPLE = _lib.SPH_SAMPLE


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _require_gpu(name: str, t: torch.Tensor) -> None:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dim() >= 1 and t.numel() > 0 and t.stride(-1) != 1:
        raise ValueError(f"{name} must be contiguous along its last dimension")


def _as_bits16(t: torch.Tensor) -> torch.Tensor:
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return t
    raise TypeError(f"expected bf16 (or its 16-bit patterns), got {t.dtype}")


class Subset:
    """Device plan of a vocabulary subset V_l (strictly ascending ids)."""

    def __init__(self, ids=None, vocab: int = 0, full: bool = False, device=None):
        lib = _lib.load()
        self._lib = lib
        self.handle = ctypes_vp()
        dev = torch.device("cuda") if device is None else torch.device(device)
        with torch.cuda.device(dev):
            stream = _stream_handle(dev)
            if full:
                check(lib.sph_subset_create_full(int(vocab), stream, self.handle))
            else:
                import numpy as np
                host = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
                check(lib.sph_subset_create(host.ctypes.data, host.size, int(vocab), stream,
                                            self.handle))
        n = _lib.c_i64()
        v = _lib.c_i64()
        check(lib.sph_subset_size(self.handle, n, v))
        self.n, self.vocab = n.value, v.value
        self.device = dev

    def device_ids_ptr(self) -> int:
        p = _lib.c_vp()
        check(self._lib.sph_subset_device_ids(self.handle, p))
        return p.value

    def close(self) -> None:
        if self.handle is not None and self.handle.value:
            self._lib.sph_subset_destroy(self.handle)
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class GcmKey:
    """Device AES-GCM key (16- or 32-byte key) for sealing payload rows (eq. 19)."""

    def __init__(self, key: bytes, device=None):
        import ctypes
        lib = _lib.load()
        self._lib = lib
        self.handle = ctypes_vp()
        key = bytes(key)
        buf = ctypes.create_string_buffer(key, len(key))
        dev = torch.device("cuda") if device is None else torch.device(device)
        with torch.cuda.device(dev):
            check(lib.sph_gcm_key_create(ctypes.addressof(buf), len(key), _stream_handle(dev),
                                         self.handle))
        ctypes.memset(buf, 0, len(key))
        self.device = dev

    def close(self) -> None:
        if self.handle is not None and self.handle.value:
            self._lib.sph_gcm_key_destroy(self.handle)
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def gcm_workspace(rows: int, row_bytes: int) -> int:
    return int(_lib.load().sph_gcm_workspace(int(rows), int(row_bytes)))


def _rows_u8(t: torch.Tensor, name: str):
    _require_gpu(name, t)
    if t.dim() != 2 or (t.shape[0] > 0 and t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"{name}: expected a 2-D tensor whose rows are contiguous")
    rows = t.shape[0]
    row_bytes = t.shape[1] * t.element_size()
    ld = t.stride(0) * t.element_size() if rows > 0 else row_bytes
    return rows, row_bytes, ld


def _check_bytes(t: torch.Tensor, name: str, shape) -> None:
    _require_gpu(name, t)
    if t.dtype != torch.uint8 or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous uint8 {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")


def _check_msg_args(rows: int, iv: torch.Tensor, aad: Optional[torch.Tensor]) -> None:
    _check_bytes(iv, "iv", (rows, 12))
    if aad is not None:
        _require_gpu("aad", aad)
        if aad.dtype != torch.uint8 or aad.dim() != 2 or aad.shape[0] != rows or \
                (aad.shape[1] > 1 and aad.stride(1) != 1):
            raise ValueError("aad: expected uint8 [rows, a] with contiguous rows")


def gcm_seal(key: GcmKey, pt: torch.Tensor, iv: torch.Tensor, aad: Optional[torch.Tensor] = None,
             out=None, workspace: Optional[torch.Tensor] = None):
    """Seal each row of pt (a 2-D device tensor; rows are the messages) under
    iv uint8 [rows, 12] and aad uint8 [rows, a].  Returns (ct uint8 [rows,
    row_bytes], tag uint8 [rows, 16])."""
    lib = _lib.load()
    rows, row_bytes, ld = _rows_u8(pt, "pt")
    _check_msg_args(rows, iv, aad)
    dev = pt.device
    if out is None:
        ct = torch.empty((rows, row_bytes), dtype=torch.uint8, device=dev)
        tag = torch.empty((rows, 16), dtype=torch.uint8, device=dev)
    else:
        ct, tag = out
    na = 0 if aad is None else aad.shape[1]
    if workspace is None:
        workspace = torch.empty(max(gcm_workspace(rows, row_bytes), 1), dtype=torch.uint8, device=dev)
    check(lib.sph_gcm_seal(key.handle, pt.data_ptr(), ld, rows, row_bytes, iv.data_ptr(),
                           _ptr(aad), aad.stride(0) if aad is not None else 0, na,
                           ct.data_ptr(), ct.stride(0) * ct.element_size() if rows > 0 else row_bytes,
                           tag.data_ptr(), workspace.data_ptr(), workspace.numel(),
                           _stream_handle(dev)))
    return ct, tag


def gcm_open(key: GcmKey, ct: torch.Tensor, iv: torch.Tensor, tag: torch.Tensor,
             aad: Optional[torch.Tensor] = None, out=None, workspace: Optional[torch.Tensor] = None):
    """Open each row of ct; returns (pt uint8 [rows, row_bytes], ok int32
    [rows]): ok[m] = 1 when row m's tag verifies (use no row with ok 0)."""
    lib = _lib.load()
    rows, row_bytes, ld = _rows_u8(ct, "ct")
    _check_msg_args(rows, iv, aad)
    _check_bytes(tag, "tag", (rows, 16))
    dev = ct.device
    if out is None:
        pt = torch.empty((rows, row_bytes), dtype=torch.uint8, device=dev)
        ok = torch.empty((rows,), dtype=torch.int32, device=dev)
    else:
        pt, ok = out
    na = 0 if aad is None else aad.shape[1]
    if workspace is None:
        workspace = torch.empty(max(gcm_workspace(rows, row_bytes), 1), dtype=torch.uint8, device=dev)
    check(lib.sph_gcm_open(key.handle, ct.data_ptr(), ld, rows, row_bytes, iv.data_ptr(),
                           _ptr(aad), aad.stride(0) if aad is not None else 0, na, tag.data_ptr(),
                           pt.data_ptr(), pt.stride(0) * pt.element_size() if rows > 0 else row_bytes,
                           ok.data_ptr(), workspace.data_ptr(), workspace.numel(),
                           _stream_handle(dev)))
    return pt, ok


def _segment_array(ins, outs, rows: int, what: str):
    if not 1 <= len(ins) <= _lib.SPH_GCM_MAX_SEGMENTS or len(outs) != len(ins):
        raise ValueError(f"{what}: 1..{_lib.SPH_GCM_MAX_SEGMENTS} segments with one output each")
    arr = (_lib.GcmSegment * len(ins))()
    total = 0
    for k, (a, b) in enumerate(zip(ins, outs)):
        r, nb, ld = _rows_u8(a, f"{what} segment {k}")
        ro, nbo, ldo = _rows_u8(b, f"{what} output {k}")
        if r != rows or ro != rows or nbo != nb:
            raise ValueError(f"{what}: segment {k} is {r} x {nb} bytes, output {ro} x {nbo}, rows {rows}")
        arr[k] = _lib.GcmSegment(a.data_ptr(), ld, b.data_ptr(), ldo, nb)
        total += nb
    return arr, total


def gcm_seal_segments(key: GcmKey, segments, iv: torch.Tensor, aad: Optional[torch.Tensor] = None,
                      out=None, tag: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None):
    """Seal messages that are the concatenation of row m of each tensor in
    `segments` (2-D device tensors with the same number of rows, e.g. the
    payload codes and their scales).  Returns ([ct per segment, uint8, same
    rows x bytes], tag uint8 [rows, 16]); pass `out` (a list of uint8
    tensors, may be the inputs themselves) to write in place."""
    lib = _lib.load()
    segments = list(segments)
    rows = segments[0].shape[0] if segments else 0
    dev = segments[0].device if segments else torch.device("cuda")
    if out is None:
        out = [torch.empty((rows, _rows_u8(a, "segment")[1]), dtype=torch.uint8, device=dev)
               for a in segments]
    arr, total = _segment_array(segments, list(out), rows, "gcm_seal_segments")
    _check_msg_args(rows, iv, aad)
    if tag is None:
        tag = torch.empty((rows, 16), dtype=torch.uint8, device=dev)
    _check_bytes(tag, "tag", (rows, 16))
    na = 0 if aad is None else aad.shape[1]
    if workspace is None:
        workspace = torch.empty(max(gcm_workspace(rows, total), 1), dtype=torch.uint8, device=dev)
    check(lib.sph_gcm_seal_segments(key.handle, arr, len(segments), rows, iv.data_ptr(), _ptr(aad),
                                    aad.stride(0) if aad is not None else 0, na, tag.data_ptr(),
                                    workspace.data_ptr(), workspace.numel(), _stream_handle(dev)))
    return list(out), tag


def gcm_open_segments(key: GcmKey, segments, iv: torch.Tensor, tag: torch.Tensor,
                      aad: Optional[torch.Tensor] = None, out=None, ok: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None):
    """Open messages sealed by gcm_seal_segments; returns ([pt per segment],
    ok int32 [rows]) with ok[m] = 1 when message m's tag verifies."""
    lib = _lib.load()
    segments = list(segments)
    rows = segments[0].shape[0] if segments else 0
    dev = segments[0].device if segments else torch.device("cuda")
    if out is None:
        out = [torch.empty((rows, _rows_u8(a, "segment")[1]), dtype=torch.uint8, device=dev)
               for a in segments]
    arr, total = _segment_array(segments, list(out), rows, "gcm_open_segments")
    _check_msg_args(rows, iv, aad)
    _check_bytes(tag, "tag", (rows, 16))
    if ok is None:
        ok = torch.empty((rows,), dtype=torch.int32, device=dev)
    elif ok.dtype != torch.int32 or tuple(ok.shape) != (rows,) or not ok.is_cuda:
        raise ValueError(f"ok: expected int32 ({rows},) on the GPU")
    na = 0 if aad is None else aad.shape[1]
    if workspace is None:
        workspace = torch.empty(max(gcm_workspace(rows, total), 1), dtype=torch.uint8, device=dev)
    check(lib.sph_gcm_open_segments(key.handle, arr, len(segments), rows, iv.data_ptr(), _ptr(aad),
                                    aad.stride(0) if aad is not None else 0, na, tag.data_ptr(),
                                    ok.data_ptr(), workspace.data_ptr(), workspace.numel(),
                                    _stream_handle(dev)))
    return list(out), ok


def ctypes_vp():
    return _lib.c_vp()


def cloud_partial_workspace(M: int, subset: Subset) -> int:
    return int(_lib.load().sph_cloud_partial_workspace(int(M), subset.handle))


def fuse_verify_workspace(M: int, subset: Subset, mode: int = GREEDY) -> int:
    return int(_lib.load().sph_fuse_verify_workspace(int(M), subset.handle, int(mode)))


def payload_code_bytes(n: int, bits: int = 8) -> int:
    """Bytes of one payload row's codes (include/sph.h)."""
    return int(_lib.load().sph_payload_code_bytes(int(n), int(bits)))


def payload_scale_count(n: int, block: int = 0) -> int:
    """Scales of one payload row (include/sph.h)."""
    return int(_lib.load().sph_payload_scale_count(int(n), int(block)))


def cloud_partial(h_cloud: torch.Tensor, w_cloud: torch.Tensor, subset: Subset, clip_c: float,
                  w_row_scale: Optional[torch.Tensor] = None, bias: Optional[torch.Tensor] = None,
                  want_z: bool = False, workspace: Optional[torch.Tensor] = None, out=None,
                  bits: int = 8, block: int = 0):
    """Cloud half: returns (q, scale, z fp32 [M, n] or None).

    h_cloud: bf16 [M, d_cloud] view (rows may be strided, e.g. h[:, d_end:]).
    w_cloud: bf16 [V, d_cloud] or fp8 E4M3 (torch.float8_e4m3fn / uint8) with
    w_row_scale fp32 [V].
    Payload format (bits, block): q is int8 [M, n] for 8-bit codes, uint8
    [M, ceil(n/2)] (two codes per byte) for 4-bit codes; scale is fp32 [M]
    for one scale per row (block 0), else [M, ceil(n / block)].
    """
    lib = _lib.load()
    _require_gpu("h_cloud", h_cloud)
    _require_gpu("w_cloud", w_cloud)
    h_cloud = _as_bits16(h_cloud)
    if w_cloud.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        wtype = _lib.SPH_W_BF16
    elif w_cloud.dtype in (torch.float8_e4m3fn, torch.uint8):
        wtype = _lib.SPH_W_FP8_E4M3
    else:
        raise TypeError(f"unsupported weight dtype {w_cloud.dtype}")
    M, d_cloud = h_cloud.shape
    dev = h_cloud.device
    if out is None:
        nb = payload_scale_count(subset.n, block)
        if bits == 8:
            q = torch.empty((M, subset.n), dtype=torch.int8, device=dev)
        else:
            q = torch.empty((M, max(payload_code_bytes(subset.n, bits), 0)), dtype=torch.uint8, device=dev)
        scale = torch.empty((M,) if block == 0 else (M, max(nb, 0)), dtype=torch.float32, device=dev)
        z = torch.empty((M, subset.n), dtype=torch.float32, device=dev) if want_z else None
    else:
        q, scale, z = out
    need = cloud_partial_workspace(M, subset)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    check(lib.sph_cloud_partial_fmt(
        h_cloud.data_ptr(), h_cloud.stride(0) if M > 0 else d_cloud, M, d_cloud,
        w_cloud.data_ptr(), w_cloud.stride(0), wtype, _ptr(w_row_scale),
        _ptr(bias), subset.handle, float(clip_c), int(bits), int(block),
        q.data_ptr(), scale.data_ptr(), _ptr(z),
        workspace.data_ptr(), workspace.numel(), _stream_handle(dev)))
    return q, scale, z


NOALLOC_SCRATCH_BYTES = 16 << 20


def cloud_partial_noalloc(h_cloud: torch.Tensor, w_cloud: torch.Tensor, subset: Subset,
                          clip_c: float, out, w_row_scale: Optional[torch.Tensor] = None,
                          bias: Optional[torch.Tensor] = None, bits: int = 8, block: int = 0):
    """cloud_partial without a workspace: the library's static device scratch
    (NOALLOC_SCRATCH_BYTES per GPU) stands in for it.  `out` = (q, scale, z or
    None) must be given; nothing is allocated.  Calls that overlap on one GPU
    race (they share the scratch)."""
    lib = _lib.load()
    _require_gpu("h_cloud", h_cloud)
    _require_gpu("w_cloud", w_cloud)
    h_cloud = _as_bits16(h_cloud)
    if w_cloud.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        wtype = _lib.SPH_W_BF16
    elif w_cloud.dtype in (torch.float8_e4m3fn, torch.uint8):
        wtype = _lib.SPH_W_FP8_E4M3
    else:
        raise TypeError(f"unsupported weight dtype {w_cloud.dtype}")
    M, d_cloud = h_cloud.shape
    q, scale, z = out
    check(lib.sph_cloud_partial_noalloc(
        h_cloud.data_ptr(), h_cloud.stride(0) if M > 0 else d_cloud, M, d_cloud,
        w_cloud.data_ptr(), w_cloud.stride(0), wtype, _ptr(w_row_scale),
        _ptr(bias), subset.handle, float(clip_c), int(bits), int(block),
        q.data_ptr(), scale.data_ptr(), _ptr(z), _stream_handle(h_cloud.device)))
    return q, scale, z


def fuse_verify(q: torch.Tensor, scale: torch.Tensor, h_end: Optional[torch.Tensor],
                w_end: Optional[torch.Tensor], subset: Subset, n_sessions: int,
                rows_per_session: int, drafts: Optional[torch.Tensor], mode: int = GREEDY,
                temperature: float = 1.0, top_p: float = 1.0, seed: int = 0,
                want_fused: bool = False, workspace: Optional[torch.Tensor] = None, out=None,
                bits: int = 8, block: int = 0):
    """Endpoint half: returns (tokens int32 [M], accept_len int32 [S], fused fp32 or None).
    (q, scale) is a payload of cloud_partial in format (bits, block)."""
    lib = _lib.load()
    dev = q.device
    M = int(n_sessions) * int(rows_per_session)
    if h_end is not None and h_end.shape[1] > 0:
        _require_gpu("h_end", h_end)
        _require_gpu("w_end", w_end)
        h_end = _as_bits16(h_end)
        w_end = _as_bits16(w_end)
        d_end = h_end.shape[1]
        hp, ldh, wp, ldw = h_end.data_ptr(), h_end.stride(0), w_end.data_ptr(), w_end.stride(0)
    else:
        d_end, hp, ldh, wp, ldw = 0, None, 0, None, 0
    if out is None:
        tokens = torch.empty((M,), dtype=torch.int32, device=dev)
        accept = torch.empty((int(n_sessions),), dtype=torch.int32, device=dev)
        fused = torch.empty((M, subset.n), dtype=torch.float32, device=dev) if want_fused else None
    else:
        tokens, accept, fused = out
    need = fuse_verify_workspace(M, subset, mode)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    check(lib.sph_fuse_verify_fmt(
        q.data_ptr(), scale.data_ptr(), int(bits), int(block), hp, ldh, d_end, wp, ldw, subset.handle,
        int(n_sessions), int(rows_per_session), _ptr(drafts),
        int(mode), float(temperature), float(top_p), int(seed) & 0xFFFFFFFFFFFFFFFF,
        tokens.data_ptr(), accept.data_ptr(), _ptr(fused),
        workspace.data_ptr(), workspace.numel(), _stream_handle(dev)))
    return tokens, accept, fused


def hidden_quantize(h: torch.Tensor, out=None):
    """Per-row int8 codes of bf16 hidden rows h [M, d] (rows may be strided):
    returns (codes int8 [M, d], scales fp32 [M])."""
    lib = _lib.load()
    _require_gpu("h", h)
    h = _as_bits16(h)
    M, d = h.shape
    if out is None:
        hq = torch.empty((M, d), dtype=torch.int8, device=h.device)
        hs = torch.empty((M,), dtype=torch.float32, device=h.device)
    else:
        hq, hs = out
    check(lib.sph_hidden_quantize(h.data_ptr(), h.stride(0) if M > 0 else d, M, d, hq.data_ptr(),
                                  hq.stride(0) if M > 0 else d, hs.data_ptr(),
                                  _stream_handle(h.device)))
    return hq, hs


def fuse_verify_hq_workspace(M: int, d_end: int, subset: Subset, mode: int = GREEDY) -> int:
    return int(_lib.load().sph_fuse_verify_hq_workspace(int(M), int(d_end), subset.handle, int(mode)))


def fuse_verify_hq(q: torch.Tensor, scale: torch.Tensor, hq: torch.Tensor, h_scale: torch.Tensor,
                   d_end: int, w_end: Optional[torch.Tensor], subset: Subset, n_sessions: int,
                   rows_per_session: int, drafts: Optional[torch.Tensor], mode: int = GREEDY,
                   temperature: float = 1.0, top_p: float = 1.0, seed: int = 0,
                   want_fused: bool = False, workspace: Optional[torch.Tensor] = None, out=None,
                   bits: int = 8, block: int = 0):
    """Endpoint half on hidden-state codes: hq int8 [M, >= d_end] and h_scale
    fp32 [M] from hidden_quantize; the first d_end columns enter eq. 11.
    Returns (tokens int32 [M], accept_len int32 [S], fused fp32 or None)."""
    lib = _lib.load()
    dev = q.device
    M = int(n_sessions) * int(rows_per_session)
    d_end = int(d_end)
    if d_end > 0:
        _require_gpu("hq", hq)
        if hq.dtype != torch.int8 or hq.dim() != 2 or hq.shape[0] != M or hq.shape[1] < d_end or \
                hq.stride(1) != 1:
            raise ValueError(f"hq: expected int8 [{M}, >= {d_end}] with contiguous rows")
        if h_scale.dtype != torch.float32 or tuple(h_scale.shape) != (M,) or not h_scale.is_contiguous():
            raise ValueError(f"h_scale: expected contiguous float32 [{M}]")
        _require_gpu("w_end", w_end)
        w_end = _as_bits16(w_end)
        hp, ldh, sp = hq.data_ptr(), hq.stride(0), h_scale.data_ptr()
        wp, ldw = w_end.data_ptr(), w_end.stride(0)
    else:
        hp, ldh, sp, wp, ldw = None, 0, None, None, 0
    if out is None:
        tokens = torch.empty((M,), dtype=torch.int32, device=dev)
        accept = torch.empty((int(n_sessions),), dtype=torch.int32, device=dev)
        fused = torch.empty((M, subset.n), dtype=torch.float32, device=dev) if want_fused else None
    else:
        tokens, accept, fused = out
    need = fuse_verify_hq_workspace(M, d_end, subset, mode)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    check(lib.sph_fuse_verify_hq(
        q.data_ptr(), scale.data_ptr(), int(bits), int(block), hp, ldh, sp, d_end, wp, ldw,
        subset.handle, int(n_sessions), int(rows_per_session), _ptr(drafts),
        int(mode), float(temperature), float(top_p), int(seed) & 0xFFFFFFFFFFFFFFFF,
        tokens.data_ptr(), accept.data_ptr(), _ptr(fused),
        workspace.data_ptr(), workspace.numel(), _stream_handle(dev)))
    return tokens, accept, fused


def debug_sync(enable: Optional[bool] = None) -> bool:
    """Switch the library's debug synchronisation (a stream synchronisation
    and error check after every kernel launch region) on or off; None only
    queries.  Returns the previous state."""
    return bool(_lib.load().sph_debug_sync(-1 if enable is None else int(bool(enable))))


def trace_start(capacity: int) -> None:
    """Record HIP events around the next `capacity` kernel launches."""
    check(_lib.load().sph_trace_start(int(capacity)))


def trace_collect(capacity: int):
    """Stop tracing and return [(kernel name, milliseconds)] in launch order."""
    import ctypes
    lib = _lib.load()
    recs = (_lib.TraceRecord * int(capacity))()
    n = ctypes.c_int(0)
    check(lib.sph_trace_stop(recs, int(capacity), n))
    return [(recs[i].kernel.decode(), float(recs[i].ms)) for i in range(min(n.value, capacity))]


def probe_read(buf: torch.Tensor, sink: torch.Tensor) -> None:
    """Enqueue one streaming read of all of `buf` (measurement helper of
    include/sph_probe.h); time it with events on the current stream."""
    _require_gpu("buf", buf)
    _require_gpu("sink", sink)
    check(_lib.load().sph_probe_read(buf.data_ptr(), buf.numel() * buf.element_size(),
                                     sink.data_ptr(), _stream_handle(buf.device)))


def probe_mfma(iters: int, sink: torch.Tensor) -> float:
    """Enqueue one bf16 MFMA loop of `iters` iterations (measurement helper of
    include/sph_probe.h) and return its floating-point operation count."""
    import ctypes
    _require_gpu("sink", sink)
    flops = ctypes.c_double(0.0)
    check(_lib.load().sph_probe_mfma(int(iters), sink.data_ptr(), _stream_handle(sink.device),
                                     ctypes.byref(flops)))
    return flops.value
