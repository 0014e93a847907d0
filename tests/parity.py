"""Staged parity between the HIP library and the CPU oracle.

Tolerance (fp32 partial logits): |dz| <= 1e-3 * sum_i |h_i w_i| + 1e-5 per
element.  Integer results (int8 codes, token ids, accepted lengths) must be
bit-exact except where that tolerance can legitimately flip them; the
exemption of each stage is computed from the tolerance, element by element.

Stages:
  A  GPU fp32 partials vs oracle partials, elementwise within tolerance.
  B  the oracle's clip+quantiser applied to the GPU's own partials must give
     the GPU's codes and scales bit for bit.
  C  GPU codes vs oracle codes: equal unless the oracle's pre-rounding value
     t lies within the propagated tolerance of a rounding boundary.
  D  the oracle's endpoint steps fed the GPU's payload: fused logits within
     tolerance, tokens equal unless a competitor lies within the combined
     error bound, accepted lengths equal unless an exempt row decides them.
  E  the whole GPU pipeline vs the whole oracle pipeline, with the code and
     scale differences folded into the per-element bound.
"""

from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2607_13093_amd as sph

REL = 1e-3
ABS = 1e-5
ULP = 2.0 ** -23


def tol_of(absdot):
    return REL * absdot + ABS


# ---------------------------------------------------------------------------
# device plumbing
# ---------------------------------------------------------------------------

def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.view(dtype)
    return t.cuda()


class DeviceWorkload:
    """A workload's tensors on the GPU plus its subset plan."""

    def __init__(self, wl, h_bits=None, w_end_bits=None, w_cloud_bits=None):
        cfg = wl.cfg
        self.wl, self.cfg = wl, cfg
        self.h = to_dev(wl.h_bits if h_bits is None else h_bits, torch.bfloat16)
        self.w_end = to_dev(wl.w_end_bits if w_end_bits is None else w_end_bits, torch.bfloat16)
        if cfg.wtype == "bf16":
            self.w_cloud = to_dev(wl.w_cloud_bits if w_cloud_bits is None else w_cloud_bits,
                                  torch.bfloat16)
            self.w_scale = None
        else:
            self.w_cloud = to_dev(wl.w_cloud_codes, torch.uint8)
            self.w_scale = to_dev(wl.w_cloud_scale)
        self.bias = None if wl.bias is None else to_dev(wl.bias)
        if wl.full_vocab:
            self.subset = sph.Subset(vocab=cfg.vocab, full=True)
        else:
            self.subset = sph.Subset(wl.subset, vocab=cfg.vocab)

    def cloud(self, rows=None, want_z=True, bits=8, block=0):
        de = self.cfg.d_end
        h = self.h if rows is None else self.h[rows[0]:rows[1]]
        q, s, z = sph.cloud_partial(h[:, de:], self.w_cloud, self.subset, self.cfg.clip_c,
                                    w_row_scale=self.w_scale, bias=self.bias, want_z=want_z,
                                    bits=bits, block=block)
        return q, s, z

    def fuse(self, q, s, drafts, want_fused=True, n_sessions=None, h=None, bits=8, block=0):
        cfg = self.cfg
        de = cfg.d_end
        h = self.h if h is None else h
        S = cfg.sessions if n_sessions is None else n_sessions
        d = None if drafts is None else to_dev(np.asarray(drafts, np.int32))
        mode = sph.GREEDY if cfg.mode == "greedy" else sph.SAMPLE
        return sph.fuse_verify(q, s, h[:, :de], self.w_end, self.subset, S,
                               cfg.rows_per_session, d, mode=mode, temperature=cfg.temperature,
                               top_p=cfg.top_p, seed=cfg.philox_seed, want_fused=want_fused,
                               bits=bits, block=block)


def host(t):
    return None if t is None else t.cpu().numpy()


# ---------------------------------------------------------------------------
# stage checks
# ---------------------------------------------------------------------------

def stage_a(z_gpu, orc):
    tol = tol_of(orc["absdot"])
    dz = np.abs(z_gpu.astype(np.float64) - orc["z"].astype(np.float64))
    bad = dz > tol
    assert not bad.any(), f"stage A: {bad.sum()} partials outside tolerance, worst {dz.max():.3e}"
    return {"max_abs_err": float(dz.max()) if dz.size else 0.0,
            "max_err_over_eps_sum": float((dz / (2.0 ** -24 * orc["absdot"] + 1e-30)).max()) if dz.size else 0.0}


def stage_b(z_gpu, q_gpu, s_gpu, clip_c):
    ref = oracle.clip_quantize(z_gpu, clip_c)
    np.testing.assert_array_equal(ref["scale"].view(np.uint32), s_gpu.view(np.uint32),
                                  err_msg="stage B: scales differ from the quantiser applied to the GPU partials")
    np.testing.assert_array_equal(ref["q"], q_gpu,
                                  err_msg="stage B: codes differ from the quantiser applied to the GPU partials")


def stage_c(q_gpu, s_gpu, orc):
    tol = tol_of(orc["absdot"])
    y, a, s, t = orc["y"], orc["amax"].astype(np.float64), orc["scale"].astype(np.float64), orc["t"]
    M = y.shape[0]
    am = np.argmax(np.abs(y), axis=1)
    tol_a = tol[np.arange(M), am]
    dq = np.abs(q_gpu.astype(np.int32) - orc["q"].astype(np.int32))
    assert dq.max(initial=0) <= 1, "stage C: a code differs by more than one step"
    with np.errstate(divide="ignore", invalid="ignore"):
        bound = (tol + np.abs(y) * (tol_a / a)[:, None]) / s[:, None]
        frac = t.astype(np.float64) - np.floor(t.astype(np.float64))
        dist = np.abs(frac - 0.5)
        exempt = dist <= bound
        exempt[a == 0] = True
        ds = np.abs(s_gpu.astype(np.float64) - s)
        ok_s = (ds <= s * (tol_a / a) + s * ULP) | (a == 0)
    assert ok_s.all(), "stage C: scale outside the propagated tolerance"
    mism = dq > 0
    assert not (mism & ~exempt).any(), f"stage C: {int((mism & ~exempt).sum())} non-exempt code mismatches"
    return {"code_mismatch": int(mism.sum()), "code_exempt": int(exempt.sum()), "codes": int(dq.size)}


def stage_b_fmt(z_gpu, payload_gpu, s_gpu, clip_c, bits, block):
    """Stage B for a payload format: the oracle's quantiser of the GPU's own
    partials, packed, must equal the GPU's payload byte for byte (padding
    nibble included) and its scales bit for bit.  Returns the GPU codes."""
    ref = oracle.clip_quantize_fmt(z_gpu, clip_c, bits, block)
    M, n = z_gpu.shape
    np.testing.assert_array_equal(ref["scale"].view(np.uint32), s_gpu.reshape(M, -1).view(np.uint32),
                                  err_msg="stage B: scales differ from the quantiser applied to the GPU partials")
    np.testing.assert_array_equal(oracle.pack_codes(ref["q"], bits), payload_gpu,
                                  err_msg="stage B: payload bytes differ from the packed oracle codes")
    return oracle.unpack_codes(payload_gpu, n, bits)


def stage_c_fmt(q_gpu, s_gpu, orc_fmt, absdot, block):
    """Stage C for a payload format (q_gpu: unpacked codes).  A block's
    maximum moves by at most the largest tolerance of its elements, so its
    scale by that much over qmax."""
    tol = tol_of(absdot)
    y, t = orc_fmt["y"], orc_fmt["t"].astype(np.float64)
    a, s = orc_fmt["amax"].astype(np.float64), orc_fmt["scale"].astype(np.float64)
    M, n = y.shape
    nb = a.shape[1]
    width = n if block == 0 else block
    tol_a = np.zeros((M, nb))
    for k in range(nb):
        seg = tol[:, k * width:(k + 1) * width]
        if seg.shape[1]:
            tol_a[:, k] = seg.max(axis=1)
    cols = block_cols(n, block)
    dq = np.abs(q_gpu.astype(np.int32) - orc_fmt["q"].astype(np.int32))
    assert dq.max(initial=0) <= 1, "stage C: a code differs by more than one step"
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = tol_a / a
        bound = (tol + np.abs(y) * rel[:, cols]) / s[:, cols]
        dist = np.abs(t - np.floor(t) - 0.5)
        exempt = (dist <= bound) | (a[:, cols] == 0)
        ds = np.abs(s_gpu.reshape(M, nb).astype(np.float64) - s)
        ok_s = (ds <= s * rel + s * ULP) | (a == 0)
    assert ok_s.all(), "stage C: scale outside the propagated tolerance"
    mism = dq > 0
    assert not (mism & ~exempt).any(), f"stage C: {int((mism & ~exempt).sum())} non-exempt code mismatches"
    return {"code_mismatch": int(mism.sum()), "code_exempt": int(exempt.sum()), "codes": int(dq.size)}


def exempt_rows(f_ref, bound):
    """Rows whose argmax may legitimately move: some competitor j lies within
    bound[j*] + bound[j] of the reference maximum f_ref[j*]."""
    f = f_ref.astype(np.float64)
    jstar = np.argmax(f_ref, axis=1)
    r = np.arange(f.shape[0])
    slack = bound[r, jstar][:, None] + bound - (f[r, jstar][:, None] - f)
    slack[r, jstar] = -np.inf
    return (slack >= 0).any(axis=1)


def check_tokens_and_accept(tok_gpu, acc_gpu, ref_tok, ref_acc, exempt, subset, S, R,
                            f_ref, bound, drafts):
    """Tokens: in S always; equal to the reference outside exempt rows; on an
    exempt row that differs, the GPU's pick j must still be a near-maximum of
    the reference logits, f_ref[j*] - f_ref[j] <= bound[j*] + bound[j] (what
    the GPU's elementwise error bound allows, and nothing more).
    Accept lengths: the GPU's must equal the verification rule applied to the
    GPU's own tokens in every session, and the oracle's where no exempt row
    among r <= a decides it."""
    subset = np.asarray(subset)
    assert np.all(np.isin(tok_gpu, subset)), "token outside the subset"
    bad = (tok_gpu != ref_tok) & ~exempt
    assert not bad.any(), f"{bad.sum()} non-exempt token mismatches (rows {np.flatnonzero(bad)[:8]})"
    M = tok_gpu.shape[0]
    r = np.arange(M)
    f = f_ref.astype(np.float64)
    jstar = np.argmax(f_ref, axis=1)
    pos = np.searchsorted(subset, tok_gpu)
    gap = f[r, jstar] - f[r, pos]
    near = gap <= bound[r, jstar] + bound[r, pos]
    diff = tok_gpu != ref_tok
    assert near[diff].all(), (f"exempt rows {np.flatnonzero(diff & ~near)[:8]}: the GPU's token is not "
                              f"within the error bound of the row maximum")
    own = oracle.accept_lengths(tok_gpu, drafts, S, R)
    np.testing.assert_array_equal(acc_gpu, own, err_msg="accept lengths differ from the rule "
                                                        "applied to the GPU's own tokens")
    ex = exempt.reshape(S, R)
    for s in range(S):
        a = int(ref_acc[s])
        if ex[s, :a + 1].any():
            continue
        assert acc_gpu[s] == a, f"accept length of session {s}: gpu {acc_gpu[s]} oracle {a}"
    return {"token_mismatch": int(diff.sum()), "token_exempt_rows": int(exempt.sum())}


def block_cols(n, block):
    """Scale index of every subset position: 0 for one scale per row."""
    return np.zeros(n, np.int64) if block == 0 else np.arange(n) // block


def _fuse(q, s, z_e, block):
    if s.ndim == 1:
        return oracle.fuse_masked(q, s, z_e)
    return oracle.fuse_masked_fmt(q, s, z_e, block)


def stage_d_greedy(q_gpu, s_gpu, f_gpu, tok_gpu, acc_gpu, wl, drafts, rows=None, block=0):
    """q_gpu: int8 codes [M, n]; s_gpu: scales [M] (one per row) or [M, nb]."""
    cfg = wl.cfg
    h = wl.h_bits if rows is None else wl.h_bits[rows[0]:rows[1]]
    S = h.shape[0] // cfg.rows_per_session
    z_e, absdot = oracle.endpoint_partial_logits(h, cfg.d_end, wl.subset, wl.w_end_bits, with_abs=True)
    f_ref = _fuse(q_gpu, s_gpu, z_e, block)
    bound = tol_of(absdot) + ULP * np.abs(f_ref.astype(np.float64))
    if f_gpu is not None:
        df = np.abs(f_gpu.astype(np.float64) - f_ref.astype(np.float64))
        assert (df <= bound).all(), f"stage D: fused logits outside tolerance, worst {df.max():.3e}"
    ref_tok, _, _ = oracle.greedy_select(f_ref, wl.subset)
    ref_acc = oracle.accept_lengths(ref_tok, drafts, S, cfg.rows_per_session)
    ex = exempt_rows(f_ref, bound)
    return check_tokens_and_accept(tok_gpu, acc_gpu, ref_tok, ref_acc, ex, wl.subset, S,
                                   cfg.rows_per_session, f_ref, bound, drafts)


def stage_e_greedy(q_gpu, s_gpu, tok_gpu, acc_gpu, orc_cloud, wl, drafts, rows=None, block=0):
    cfg = wl.cfg
    h = wl.h_bits if rows is None else wl.h_bits[rows[0]:rows[1]]
    S = h.shape[0] // cfg.rows_per_session
    z_e, absdot = oracle.endpoint_partial_logits(h, cfg.d_end, wl.subset, wl.w_end_bits, with_abs=True)
    f_ref = _fuse(orc_cloud["q"], orc_cloud["scale"], z_e, block)
    ref_tok, _, _ = oracle.greedy_select(f_ref, wl.subset)
    ref_acc = oracle.accept_lengths(ref_tok, drafts, S, cfg.rows_per_session)
    # scales per subset position
    cols = block_cols(q_gpu.shape[1], block)
    s_o = orc_cloud["scale"].astype(np.float64).reshape(q_gpu.shape[0], -1)
    s_g = s_gpu.astype(np.float64).reshape(q_gpu.shape[0], -1)
    s_ref = s_o[:, cols]
    dq = np.abs(q_gpu.astype(np.float64) - orc_cloud["q"].astype(np.float64))
    ds = np.abs(s_g - s_o)[:, cols]
    bound = (dq * s_ref + np.abs(q_gpu.astype(np.float64)) * ds + tol_of(absdot)
             + ULP * np.abs(f_ref.astype(np.float64)))
    ex = exempt_rows(f_ref, bound)
    return check_tokens_and_accept(tok_gpu, acc_gpu, ref_tok, ref_acc, ex, wl.subset, S,
                                   cfg.rows_per_session, f_ref, bound, drafts)


def check_boundary_rows(tok_gpu, tok_ref, f, subset, cfg, rows, margin):
    """A row exempt in stage D (the same fused logits on both sides) may only
    differ by a decision at a boundary: the GPU's token must be one the
    oracle's sampler reaches when the cut or the draw moves by `margin`."""
    diff = np.flatnonzero(tok_gpu != tok_ref)
    if diff.size == 0:
        return
    cand = oracle.sample_candidates(f[diff], subset, cfg.temperature, cfg.top_p, cfg.philox_seed,
                                    cfg.rows_per_session, margin, row_index=np.asarray(rows)[diff])
    for m, c in zip(diff, cand):
        assert tok_gpu[m] in c, (f"row {rows[m]}: sampled {tok_gpu[m]}, oracle {tok_ref[m]}, "
                                 f"boundary candidates {c[:8]}")
