"""ctypes loader for libsph.so: symbol declarations only.

There is no fallback: if the library is missing, loading fails loudly.
"""

from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsph.so")

c_i64 = ctypes.c_int64
c_vp = ctypes.c_void_p

# name -> (restype, argtypes); mirrors include/sph.h and include/sph_probe.h
SIGNATURES = {
    "sph_abi_version": (ctypes.c_int, []),
    "sph_last_error": (ctypes.c_char_p, []),
    "sph_debug_sync": (ctypes.c_int, [ctypes.c_int]),
    "sph_subset_create": (ctypes.c_int, [c_vp, c_i64, c_i64, c_vp, ctypes.POINTER(c_vp)]),
    "sph_subset_create_full": (ctypes.c_int, [c_i64, c_vp, ctypes.POINTER(c_vp)]),
    "sph_subset_size": (ctypes.c_int, [c_vp, ctypes.POINTER(c_i64), ctypes.POINTER(c_i64)]),
    "sph_subset_device_ids": (ctypes.c_int, [c_vp, ctypes.POINTER(c_vp)]),
    "sph_subset_destroy": (None, [c_vp]),
    "sph_cloud_partial_workspace": (ctypes.c_size_t, [c_i64, c_vp]),
    "sph_fuse_verify_workspace": (ctypes.c_size_t, [c_i64, c_vp, ctypes.c_int]),
    "sph_cloud_partial": (ctypes.c_int, [
        c_vp, c_i64, c_i64, c_i64,          # h_cloud, ldh, M, d_cloud
        c_vp, c_i64, ctypes.c_int, c_vp,    # w_cloud, ldw, wtype, w_row_scale
        c_vp, c_vp, ctypes.c_float,         # bias, subset, clip_c
        c_vp, c_vp, c_vp,                   # q_out, scale_out, z_out
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_fuse_verify": (ctypes.c_int, [
        c_vp, c_vp,                         # q, scale
        c_vp, c_i64, c_i64,                 # h_end, ldh, d_end
        c_vp, c_i64, c_vp,                  # w_end, ldw, subset
        c_i64, c_i64, c_vp,                 # n_sessions, rows_per_session, drafts
        ctypes.c_int, ctypes.c_float, ctypes.c_float, ctypes.c_uint64,  # mode, temperature, top_p, seed
        c_vp, c_vp, c_vp,                   # tokens_out, accept_len_out, fused_out
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_payload_code_bytes": (c_i64, [c_i64, ctypes.c_int]),
    "sph_payload_scale_count": (c_i64, [c_i64, c_i64]),
    "sph_cloud_partial_fmt": (ctypes.c_int, [
        c_vp, c_i64, c_i64, c_i64,          # h_cloud, ldh, M, d_cloud
        c_vp, c_i64, ctypes.c_int, c_vp,    # w_cloud, ldw, wtype, w_row_scale
        c_vp, c_vp, ctypes.c_float,         # bias, subset, clip_c
        ctypes.c_int, c_i64,                # bits, block
        c_vp, c_vp, c_vp,                   # q_out, scale_out, z_out
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_cloud_partial_noalloc": (ctypes.c_int, [
        c_vp, c_i64, c_i64, c_i64,          # h_cloud, ldh, M, d_cloud
        c_vp, c_i64, ctypes.c_int, c_vp,    # w_cloud, ldw, wtype, w_row_scale
        c_vp, c_vp, ctypes.c_float,         # bias, subset, clip_c
        ctypes.c_int, c_i64,                # bits, block
        c_vp, c_vp, c_vp,                   # q_out, scale_out, z_out
        c_vp]),                             # stream
    "sph_fuse_verify_fmt": (ctypes.c_int, [
        c_vp, c_vp, ctypes.c_int, c_i64,    # q, scale, bits, block
        c_vp, c_i64, c_i64,                 # h_end, ldh, d_end
        c_vp, c_i64, c_vp,                  # w_end, ldw, subset
        c_i64, c_i64, c_vp,                 # n_sessions, rows_per_session, drafts
        ctypes.c_int, ctypes.c_float, ctypes.c_float, ctypes.c_uint64,  # mode, temperature, top_p, seed
        c_vp, c_vp, c_vp,                   # tokens_out, accept_len_out, fused_out
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_hidden_quantize": (ctypes.c_int, [
        c_vp, c_i64, c_i64, c_i64,          # h, ldh, M, d
        c_vp, c_i64, c_vp, c_vp]),          # q_out, ldq, scale_out, stream
    "sph_fuse_verify_hq_workspace": (ctypes.c_size_t, [c_i64, c_i64, c_vp, ctypes.c_int]),
    "sph_fuse_verify_hq": (ctypes.c_int, [
        c_vp, c_vp, ctypes.c_int, c_i64,    # q, scale, bits, block
        c_vp, c_i64, c_vp, c_i64,           # hq, ldhq, h_scale, d_end
        c_vp, c_i64, c_vp,                  # w_end, ldw, subset
        c_i64, c_i64, c_vp,                 # n_sessions, rows_per_session, drafts
        ctypes.c_int, ctypes.c_float, ctypes.c_float, ctypes.c_uint64,  # mode, temperature, top_p, seed
        c_vp, c_vp, c_vp,                   # tokens_out, accept_len_out, fused_out
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_gcm_key_create": (ctypes.c_int, [c_vp, ctypes.c_int, c_vp, ctypes.POINTER(c_vp)]),
    "sph_gcm_key_destroy": (None, [c_vp]),
    "sph_gcm_workspace": (ctypes.c_size_t, [c_i64, c_i64]),
    "sph_gcm_seal": (ctypes.c_int, [
        c_vp, c_vp, c_i64, c_i64, c_i64,    # key, pt, ld_pt, rows, row_bytes
        c_vp, c_vp, c_i64, c_i64,           # iv, aad, ld_aad, aad_bytes
        c_vp, c_i64, c_vp,                  # ct, ld_ct, tag
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_gcm_open": (ctypes.c_int, [
        c_vp, c_vp, c_i64, c_i64, c_i64,    # key, ct, ld_ct, rows, row_bytes
        c_vp, c_vp, c_i64, c_i64,           # iv, aad, ld_aad, aad_bytes
        c_vp, c_vp, c_i64, c_vp,            # tag, pt, ld_pt, ok_out
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_gcm_seal_segments": (ctypes.c_int, [
        c_vp, c_vp, ctypes.c_int, c_i64,    # key, segments, nseg, rows
        c_vp, c_vp, c_i64, c_i64,           # iv, aad, ld_aad, aad_bytes
        c_vp, c_vp, ctypes.c_size_t, c_vp]),  # tag, workspace, ws_bytes, stream
    "sph_gcm_open_segments": (ctypes.c_int, [
        c_vp, c_vp, ctypes.c_int, c_i64,    # key, segments, nseg, rows
        c_vp, c_vp, c_i64, c_i64,           # iv, aad, ld_aad, aad_bytes
        c_vp, c_vp,                         # tag, ok_out
        c_vp, ctypes.c_size_t, c_vp]),      # workspace, ws_bytes, stream
    "sph_trace_start": (ctypes.c_int, [ctypes.c_int]),
    "sph_trace_stop": (ctypes.c_int, [c_vp, ctypes.c_int, ctypes.POINTER(ctypes.c_int)]),
    # include/sph_probe.h
    "sph_probe_read": (ctypes.c_int, [c_vp, c_i64, c_vp, c_vp]),
    "sph_probe_mfma": (ctypes.c_int, [c_i64, c_vp, c_vp, ctypes.POINTER(ctypes.c_double)]),
}


class TraceRecord(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_char * 32), ("ms", ctypes.c_float)]


class GcmSegment(ctypes.Structure):
    """sph_gcm_segment."""
    _fields_ = [("in_", c_vp), ("ld_in", c_i64), ("out", c_vp), ("ld_out", c_i64),
                ("bytes", c_i64)]


SPH_GCM_MAX_SEGMENTS = 4


SPH_OK = 0
SPH_E_INVALID_ARG = -1
SPH_E_SUBSET = -2
SPH_E_UNSUPPORTED = -3
SPH_E_DEVICE = -4
SPH_E_WORKSPACE = -5
SPH_W_BF16 = 0
SPH_W_FP8_E4M3 = 1
SPH_GREEDY = 0
SPH_SAMPLE = 1

_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                               "(or python paper_2607_13093_amd/build.py)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


class SphError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


def check(code: int) -> None:
    if code != SPH_OK:
        raise SphError(code, load().sph_last_error().decode())
