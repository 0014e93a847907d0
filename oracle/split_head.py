"""fp64 NumPy oracle of the split LM head, its payload encoding and verification.

TEST INFRASTRUCTURE ONLY (see the package docstring): the HIP library never
imports, links or runs anything from here.

Notation follows the paper (Section 5.4): the hidden state h' is the
concatenation of h_end (the first D_end dimensions, kept on the endpoint) and
h_cloud (the remaining D_cloud dimensions); the LM-head weight is split the
same way, W_lm = [W_end; W_cloud] (eq. 10).  Weights are stored vocab-major
here, i.e. row v of an array is column v of the paper's D x V matrix.  S is
the language-restricted vocabulary subset V_l, a strictly ascending id list.

Readings where the paper is silent (each is listed with its justification in
the design notes of the repository):

* clipping is a symmetric clamp of the cloud partial logits to [-c, c];
* the b-bit quantiser Q_b of eq. 18 is per-row symmetric int8 with a dynamic
  scale s = amax/127, codes in [-127, 127], round-half-to-even, computed with
  correctly rounded fp32 division; the configurable variant takes b in {4, 8}
  (codes in [-(2^(b-1) - 1), 2^(b-1) - 1], 4-bit codes packed two per byte)
  and one scale per row or per block of subset positions;
* dequantisation and fusion are one fp32 rounding of q*s + z_end;
* greedy ties go to the lowest vocabulary id;
* sampling uses top-p nucleus selection on top of eq. 15, with the draw made
  by inverse CDF in ascending id order from a Philox4x32-10 uniform;
* draft r of a session is judged by verification row r (prefix match).
"""

from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------------------
# exact input decodings
# ---------------------------------------------------------------------------


def decode_bf16(bits) -> np.ndarray:
    """bf16 bit patterns -> exact fp64 values (a bf16 is the top half of an fp32).

    Pinned by: torch.bfloat16 -> float32 conversion of every bit pattern.
    """
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def decode_e4m3(codes) -> np.ndarray:
    """OCP 8-bit floating point, E4M3 variant -> exact fp64 values.

    Layout: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits; exponent
    field 0 encodes subnormals m/8 * 2^-6; S.1111.111 is NaN; there is no
    infinity, so the largest finite magnitude is 1.75 * 2^8 = 448.
    Pinned by: torch.float8_e4m3fn -> float32 on all 256 codes.
    """
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    normal = (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0)
    sub = (m / 8.0) * 2.0 ** -6
    val = sign * np.where(e == 0, sub, normal)
    return np.where((e == 15) & ((c & 0x7) == 7), np.nan, val)


def _cloud_rows_f64(ids, w_cloud_bits=None, w_cloud_codes=None, w_cloud_scale=None):
    """Decoded cloud weight rows W_cloud[ids] in fp64 (vocab-major)."""
    if w_cloud_bits is not None:
        return decode_bf16(w_cloud_bits[ids])
    w = decode_e4m3(w_cloud_codes[ids])
    return w * np.asarray(w_cloud_scale, dtype=np.float32)[ids].astype(np.float64)[:, None]


def _to_f32(x64: np.ndarray) -> np.ndarray:
    return np.asarray(x64, dtype=np.float64).astype(np.float32)


# ---------------------------------------------------------------------------
# eq. 9: the unsplit head (used only to pin the split)
# ---------------------------------------------------------------------------


def full_head_logits(h_bits, w_full_f64, bias=None) -> np.ndarray:
    """z = h' W_lm + b over the whole vocabulary, fp64 (eq. 9).

    ``w_full_f64`` is the complete weight [V, D] in fp64 (vocab-major).
    Brute force, small shapes only.
    """
    H = decode_bf16(h_bits)
    z = H @ np.asarray(w_full_f64, dtype=np.float64).T
    if bias is not None:
        z = z + np.asarray(bias, dtype=np.float32).astype(np.float64)[None, :]
    return z


# ---------------------------------------------------------------------------
# eq. 12 restricted to S: the cloud partial
# ---------------------------------------------------------------------------


def cloud_partial_logits(h_bits, d_end, subset, w_cloud_bits=None, w_cloud_codes=None,
                         w_cloud_scale=None, bias=None, rows=None, with_abs=False,
                         chunk=4096):
    """z_cloud[m, j] = fp32( sum_i h_cloud[m, i] * W_cloud[S_j, i] (+ b[S_j]) ).

    Eq. 12 evaluated only on the subset ids (Section 5.4: the cloud returns
    z_cloud[V_l]).  The bias is added here, on the cloud side, and nowhere
    else, so it is applied exactly once.  For fp8 weights each vocabulary
    row is decode(code) * row_scale.  The dot products are accumulated in
    fp64 (a BLAS matmul) and rounded once to fp32.

    Returns (z fp32 [M, n], absdot fp64 [M, n] or None) where absdot is
    sum_i |h_i * w_i| (+ |b|), the scale of the fp32 tolerance.
    Pinned by: the split identity against the unsplit head (eq. 9-13), the
    d_end = 0 case against torch.nn.functional.linear, the worked example.
    """
    h_bits = np.asarray(h_bits)
    if rows is not None:
        h_bits = h_bits[np.asarray(rows)]
    H = decode_bf16(h_bits[:, d_end:])
    subset = np.asarray(subset, dtype=np.int64)
    n = subset.size
    z = np.empty((H.shape[0], n), dtype=np.float32)
    absdot = np.empty((H.shape[0], n), dtype=np.float64) if with_abs else None
    for j0 in range(0, n, chunk):
        ids = subset[j0:j0 + chunk]
        W = _cloud_rows_f64(ids, w_cloud_bits, w_cloud_codes, w_cloud_scale)
        acc = H @ W.T
        if bias is not None:
            acc = acc + np.asarray(bias, dtype=np.float32)[ids].astype(np.float64)[None, :]
        z[:, j0:j0 + len(ids)] = _to_f32(acc)
        if with_abs:
            a = np.abs(H) @ np.abs(W).T
            if bias is not None:
                a = a + np.abs(np.asarray(bias, dtype=np.float32)[ids].astype(np.float64))[None, :]
            absdot[:, j0:j0 + len(ids)] = a
    return z, absdot


def clip_quantize(z, clip_c):
    """Clip the cloud partial logits and quantise each row to int8.

    Section 5.4 returns z_cloud[V_l] "after clipping, quantization and
    encryption"; eq. 18 writes the quantiser as q = Q_b(r) with b = 8 for
    logits (Section 7.3).  Reading (the paper fixes neither the clip nor
    Q_b):
        y = clamp(z, -c, c)                  (fp32)
        a = max_j |y_j|                      (exact)
        s = fp32(a / 127), s = 0 if a = 0    (correctly rounded)
        t = fp32(y / s)                      (correctly rounded)
        q = clamp(rint_half_even(t), -127, 127), q = 0 if s = 0
    Returns dict(y, amax, scale, t, q).
    Pinned by: |q*s - y| <= s/2, the code at argmax|y| is +-127, a clipped
    row has s = fp32(30/127), a zero row has s = q = 0, the worked example.
    """
    z = np.asarray(z, dtype=np.float32)
    c = np.float32(clip_c)
    y = np.minimum(np.maximum(z, -c), c)
    if y.shape[1] == 0:
        amax = np.zeros(y.shape[0], dtype=np.float32)
    else:
        amax = np.abs(y).max(axis=1).astype(np.float32)
    scale = (amax / np.float32(127.0)).astype(np.float32)
    pos = scale > 0
    t = np.zeros_like(y)
    np.divide(y, scale[:, None], out=t, where=pos[:, None])
    q = np.clip(np.rint(t), -127, 127).astype(np.int8)
    q[~pos] = 0
    return {"y": y, "amax": amax, "scale": scale, "t": t, "q": q}


def clip_quantize_fmt(z, clip_c, bits=8, block=0):
    """Clip and quantise with a configurable bit width b and scale granularity.

    Eq. 18 quantises tensor elements to a configurable bit width b, and the
    payload estimate of eq. 21 is |V_l| * b/8 bytes plus metadata.  Reading
    for b in {4, 8}: symmetric codes in [-qmax, qmax], qmax = 2^(b-1) - 1,
    with one dynamic scale per row (block = 0, the reading of clip_quantize)
    or per row and block of `block` consecutive subset positions (the last
    block of a row may be shorter):
        y = clamp(z, -c, c)                           (fp32)
        a[m, k] = max |y[m, j]| over block k          (exact)
        s[m, k] = fp32(a / qmax), 0 if a = 0          (correctly rounded)
        t = fp32(y / s[m, k(j)])                      (correctly rounded)
        q = clamp(rint_half_even(t), -qmax, qmax), 0 where s = 0
    Returns dict(y, amax [M, nb], scale [M, nb], t, q (int8 codes [M, n])).
    Pinned by: b = 8 with one scale per row reproduces clip_quantize;
    |q*s - y| <= s/2; every block's element of largest |y| gets +-qmax; a
    hand-worked 4-bit example with two blocks.
    """
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    z = np.asarray(z, dtype=np.float32)
    c = np.float32(clip_c)
    y = np.minimum(np.maximum(z, -c), c)
    M, n = y.shape
    qmax = np.float32(2 ** (bits - 1) - 1)
    width = n if block == 0 else block
    nb = 1 if block == 0 else max(1, -(-n // block))
    amax = np.zeros((M, nb), dtype=np.float32)
    for k in range(nb):
        seg = y[:, k * width:(k + 1) * width]
        if seg.shape[1]:
            amax[:, k] = np.abs(seg).max(axis=1)
    scale = (amax / qmax).astype(np.float32)
    col_scale = np.repeat(scale, width, axis=1)[:, :n] if n else np.zeros((M, 0), np.float32)
    pos = col_scale > 0
    t = np.zeros_like(y)
    np.divide(y, col_scale, out=t, where=pos)
    q = np.clip(np.rint(t), -qmax, qmax).astype(np.int8)
    q[~pos] = 0
    return {"y": y, "amax": amax, "scale": scale, "t": t, "q": q}


def pack_codes(q, bits):
    """Payload bytes of b-bit codes, row by row: b = 8 stores each code as a
    byte (two's complement); b = 4 stores code 2i in the low and code 2i+1 in
    the high nibble of byte i (two's complement nibbles; an odd row ends with
    a zero high nibble).  Returns uint8 [M, ceil(n * b / 8)].
    Pinned by: a hand-written byte pattern and the unpack round trip."""
    q = np.asarray(q, dtype=np.int8)
    if bits == 8:
        return q.view(np.uint8).copy()
    if bits != 4:
        raise ValueError("bits must be 4 or 8")
    M, n = q.shape
    nib = (q.astype(np.int16) & 0xF).astype(np.uint8)
    if n % 2:
        nib = np.concatenate([nib, np.zeros((M, 1), np.uint8)], axis=1)
    return (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)


def unpack_codes(p, n, bits):
    """Inverse of pack_codes: int8 codes [M, n]."""
    p = np.asarray(p, dtype=np.uint8)
    if bits == 8:
        return p[:, :n].view(np.int8).copy()
    lo = (p & 0xF).astype(np.int16)
    hi = (p >> 4).astype(np.int16)
    nib = np.empty((p.shape[0], 2 * p.shape[1]), np.int16)
    nib[:, 0::2] = lo
    nib[:, 1::2] = hi
    nib = np.where(nib >= 8, nib - 16, nib)
    return nib[:, :n].astype(np.int8)


def payload_bytes(n, bits, block):
    """Payload of one row (eq. 21 without transport overheads): the packed
    codes plus one fp32 scale per block (one per row for block = 0)."""
    nb = 1 if block == 0 else max(1, -(-n // block))
    return -(-n * bits // 8) + 4 * nb


# ---------------------------------------------------------------------------
# eq. 11 restricted to S: the endpoint partial
# ---------------------------------------------------------------------------


def endpoint_partial_logits(h_bits, d_end, subset, w_end_bits, rows=None, with_abs=False,
                            chunk=8192):
    """z_end[m, j] = fp32( sum_{i < D_end} h_end[m, i] * W_end[S_j, i] ).

    Eq. 11 evaluated on the subset ids (Section 5.4, the endpoint computes
    the matching local component z_end[V_l]; Algorithm 1, first step of the
    decoding loop).  fp64 accumulation, one rounding to fp32.  D_end = 0
    gives zeros.  Returns (z_end fp32 [M, n], absdot or None).
    Pinned by: the split identity and the worked example.
    """
    h_bits = np.asarray(h_bits)
    if rows is not None:
        h_bits = h_bits[np.asarray(rows)]
    H = decode_bf16(h_bits[:, :d_end])
    subset = np.asarray(subset, dtype=np.int64)
    n = subset.size
    z = np.zeros((H.shape[0], n), dtype=np.float32)
    absdot = np.zeros((H.shape[0], n), dtype=np.float64) if with_abs else None
    if d_end == 0:
        return z, absdot
    for j0 in range(0, n, chunk):
        ids = subset[j0:j0 + chunk]
        W = decode_bf16(np.asarray(w_end_bits)[ids])
        z[:, j0:j0 + len(ids)] = _to_f32(H @ W.T)
        if with_abs:
            absdot[:, j0:j0 + len(ids)] = np.abs(H) @ np.abs(W).T
    return z, absdot


# ---------------------------------------------------------------------------
# Section 5.3: the returned hidden state is quantised before it leaves the
# cloud; eq. 11 then runs on the dequantised values
# ---------------------------------------------------------------------------


def hidden_quantize(h_bits):
    """Per-row int8 quantisation of returned hidden states.

    Section 5.3 quantises (and encrypts) every tensor the cloud returns, the
    hidden state included, with the Q_b of eq. 18.  Reading (b = 8, the
    logit rule of clip_quantize without a clip, since the hidden state has
    no natural range):
        x = bf16 value (exact in fp32)
        a = max_i |x[m, i]|                    (exact)
        s = fp32(a / 127), 0 if a = 0          (correctly rounded)
        t = fp32(x / s)                        (correctly rounded)
        q = clamp(rint_half_even(t), -127, 127), 0 where s = 0
    Returns (q int8 [M, d], s fp32 [M]).
    Pinned by: a row whose maximum is 127 (s = 1, q = rint(x), ties to
    even), |q*s - x| <= s/2, +-127 at every row maximum, a zero row, and
    agreement with clip_quantize for a clip above every |x|.
    """
    x = decode_bf16(np.asarray(h_bits)).astype(np.float32)
    M = x.shape[0]
    if x.shape[1] == 0:
        return np.zeros(x.shape, np.int8), np.zeros(M, np.float32)
    amax = np.abs(x).max(axis=1)
    scale = (amax / np.float32(127.0)).astype(np.float32)
    pos = scale > 0
    t = np.zeros_like(x)
    np.divide(x, scale[:, None], out=t, where=pos[:, None])
    q = np.clip(np.rint(t), -127, 127).astype(np.int8)
    q[~pos] = 0
    return q, scale


def endpoint_partial_logits_hq(hq, h_scale, d_end, subset, w_end_bits, with_abs=False,
                               chunk=8192):
    """z_end[m, j] = fp32( sum_{i < D_end} (q[m, i] * s_m) * W_end[S_j, i] ).

    Eq. 11 on the endpoint's dequantised hidden state (the codes of
    hidden_quantize and their row scale; only the first D_end columns enter
    the sum).  q * s is exact in fp64; fp64 accumulation, one rounding.
    Returns (z_end fp32 [M, n], absdot = sum |q s| |W| or None).
    Pinned by: equality with endpoint_partial_logits when every q * s is a
    bf16 value (rows with s = 1 and s = 2^-3), and a hand-worked example.
    """
    q = np.asarray(hq, dtype=np.int8)[:, :d_end].astype(np.float64)
    s = np.asarray(h_scale, dtype=np.float32).astype(np.float64)
    H = q * s[:, None]
    subset = np.asarray(subset, dtype=np.int64)
    n = subset.size
    z = np.zeros((H.shape[0], n), dtype=np.float32)
    absdot = np.zeros((H.shape[0], n), dtype=np.float64) if with_abs else None
    if d_end == 0:
        return z, absdot
    for j0 in range(0, n, chunk):
        ids = subset[j0:j0 + chunk]
        W = decode_bf16(np.asarray(w_end_bits)[ids])
        z[:, j0:j0 + len(ids)] = _to_f32(H @ W.T)
        if with_abs:
            absdot[:, j0:j0 + len(ids)] = np.abs(H) @ np.abs(W).T
    return z, absdot


# ---------------------------------------------------------------------------
# eq. 13-14: dequantise, fuse, mask
# ---------------------------------------------------------------------------


def round_sum_to_f32(a, b) -> np.ndarray:
    """fp32 nearest (ties to even) to the exact sum a + b of fp64 values.

    The fp64 sum s = a + b may itself be rounded; TwoSum recovers the exact
    error e with s + e = a + b.  Rounding s to fp32 is then wrong only when
    s sits exactly halfway between two fp32 values and e != 0, in which case
    the exact sum lies on the side of e.
    Pinned by: exact rational arithmetic (fractions.Fraction) in a test.
    """
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    s = a + b
    bb = s - a
    e = (a - (s - bb)) + (b - bb)
    r = s.astype(np.float32)
    r64 = r.astype(np.float64)
    toward = np.where(s > r64, np.float32(np.inf), np.float32(-np.inf)).astype(np.float32)
    other = np.nextafter(r, toward)
    mid = (r64 + other.astype(np.float64)) * 0.5
    tie = (s != r64) & (s == mid) & (e != 0)
    up = np.maximum(r, other)
    down = np.minimum(r, other)
    return np.where(tie, np.where(e > 0, up, down), r).astype(np.float32)


def fuse_masked(q, scale, z_end) -> np.ndarray:
    """f[m, j] = fp32(q[m, j] * s_m + z_end[m, j]) for j in S (eq. 13-14).

    The payload is dequantised as q * s (exact in fp64) and added to the
    endpoint partial with a single rounding.  Ids outside S carry -inf in
    eq. 14; they are simply absent here, so they can never be selected.
    """
    q = np.asarray(q, dtype=np.int8).astype(np.float64)
    s = np.asarray(scale, dtype=np.float32).astype(np.float64)[:, None]
    return round_sum_to_f32(q * s, np.asarray(z_end, dtype=np.float32).astype(np.float64))


def fuse_masked_fmt(q, scale, z_end, block=0) -> np.ndarray:
    """fuse_masked with per-(row, block) scales: f[m, j] = fp32(q[m, j] *
    s[m, k(j)] + z_end[m, j]), k(j) = j // block (k = 0 for block = 0).
    Pinned by: with one scale per row it equals fuse_masked."""
    q = np.asarray(q, dtype=np.int8).astype(np.float64)
    s = np.asarray(scale, dtype=np.float32).astype(np.float64)
    n = q.shape[1]
    cols = np.zeros(n, dtype=np.int64) if block == 0 else np.arange(n) // block
    return round_sum_to_f32(q * s[:, cols], np.asarray(z_end, dtype=np.float32).astype(np.float64))


# ---------------------------------------------------------------------------
# selection
# ---------------------------------------------------------------------------


def greedy_select(f, subset):
    """Greedy token per row: the subset id with the largest fused logit.

    The zero-temperature limit of eq. 15 (Algorithm 1: the endpoint picks
    y_t from the fused, masked logits).  Ties go to the lowest id, which is
    the lowest subset position because S is ascending.  Also returns the gap
    between the best and the runner-up logit (0 on a tie, inf for |S| = 1).
    """
    f = np.asarray(f, dtype=np.float32)
    pos = np.argmax(f, axis=1)
    best = f[np.arange(f.shape[0]), pos].astype(np.float64)
    if f.shape[1] > 1:
        g = f.astype(np.float64).copy()
        g[np.arange(f.shape[0]), pos] = -np.inf
        gap = best - g.max(axis=1)
    else:
        gap = np.full(f.shape[0], np.inf)
    return np.asarray(subset, dtype=np.int32)[pos], pos, gap


_PHILOX_M0 = 0xD2511F53
_PHILOX_M1 = 0xCD9E8D57
_PHILOX_W0 = 0x9E3779B9
_PHILOX_W1 = 0xBB67AE85
_MASK32 = 0xFFFFFFFF


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11).

    Each round multiplies words 0 and 2 by the two round constants, keeps
    the 64-bit products' high and low halves, and permutes:
        (c0, c1, c2, c3) -> (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2),
                             hi(M0*c0) ^ c3 ^ k1, lo(M0*c0))
    with the key bumped by the Weyl constants between rounds.
    Pinned by: the published known-answer vectors of Philox4x32-10.
    """
    c0, c1, c2, c3 = (int(x) & _MASK32 for x in ctr)
    k0, k1 = (int(x) & _MASK32 for x in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _PHILOX_W0) & _MASK32
            k1 = (k1 + _PHILOX_W1) & _MASK32
        p0 = _PHILOX_M0 * c0
        p1 = _PHILOX_M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0, p1 & _MASK32,
                          (p0 >> 32) ^ c3 ^ k1, p0 & _MASK32)
    return c0, c1, c2, c3


def philox_uniform(seed: int, row_in_session: int, session: int) -> float:
    """u in [0, 1) for one verification row: the top 24 bits of word 0 of
    Philox4x32-10 with key (lo32(seed), hi32(seed)) and counter
    (row, session, 0, 0), times 2^-24 (exact in fp32 and fp64)."""
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    x0 = philox4x32_10((row_in_session, session, 0, 0), (seed & _MASK32, seed >> 32))[0]
    return (x0 >> 8) * 2.0 ** -24


def sample_select(f, subset, temperature, top_p, seed, rows_per_session, row_index=None):
    """Temperature + top-p sample per row (eq. 15 with a nucleus cut).

    p = softmax(f / tau) over S in fp64.  Order S by (p desc, id asc); the
    nucleus N is the shortest prefix of that order whose mass reaches top_p
    (all of S when top_p >= 1; never empty).  With u from ``philox_uniform``
    and target = u * mass(N), walk N in ascending id order and take the
    first member whose running mass exceeds the target (the last member if
    rounding leaves none).

    Row m of ``f`` is verification row row_index[m] of the batch (default m):
    its counter is (row_index[m] % R, row_index[m] // R).

    Returns (tokens int32 [M], info) where info holds, per row, the nucleus
    size, the distance of top_p from the two cumulative masses around the cut
    (inf without a cut) and the distance of the target from the nearest
    boundary of the chosen member's CDF interval, both in probability units.
    Pinned by: tau -> 0 and top_p -> 0 reduce to the greedy pick, a chi-square
    test of the draws against the exact softmax, a hand-made nucleus.
    """
    f = np.asarray(f, dtype=np.float32)
    subset = np.asarray(subset, dtype=np.int64)
    M, n = f.shape
    tau = float(np.float32(temperature))
    tp = float(np.float32(top_p))
    tokens = np.empty(M, dtype=np.int32)
    ksize = np.empty(M, dtype=np.int64)
    cut_margin = np.empty(M)
    cdf_margin = np.empty(M)
    for m in range(M):
        x = f[m].astype(np.float64)
        e = np.exp((x - x.max()) / tau)
        p = e / e.sum()
        order = np.lexsort((subset, -p))          # p descending, then id ascending
        cum = np.cumsum(p[order])
        if tp >= 1.0:
            K = n
            cut_margin[m] = np.inf
        else:
            K = min(int(np.searchsorted(cum, tp, side="left")) + 1, n)
            above = cum[K - 1] - tp
            below = tp - cum[K - 2] if K >= 2 else np.inf
            cut_margin[m] = min(above, below)
        ksize[m] = K
        members = np.sort(order[:K])              # positions in S, ascending id
        run = np.cumsum(p[members])
        mass = run[-1]
        g = m if row_index is None else int(row_index[m])
        u = philox_uniform(seed, g % rows_per_session, g // rows_per_session)
        target = u * mass
        hit = np.flatnonzero(run > target)
        i = int(hit[0]) if hit.size else K - 1
        before = run[i - 1] if i > 0 else 0.0
        cdf_margin[m] = min(target - before, run[i] - target)
        tokens[m] = subset[members[i]]
    return tokens, {"nucleus": ksize, "cut_margin": cut_margin, "cdf_margin": cdf_margin}


def sample_candidates(f, subset, temperature, top_p, seed, rows_per_session, margin,
                      row_index=None):
    """Every token the sampler of ``sample_select`` can return for a row when
    each cumulative mass it compares may be off by up to ``margin``
    (probability units): the nucleus cut may fall anywhere from the first
    prefix reaching top_p - margin to the first reaching top_p + margin, and
    for each such nucleus the draw may land on any member whose CDF interval
    comes within ``margin`` of the target (eq. 15 with the top-p cut and the
    ascending-id inverse CDF of ``sample_select``).

    Returns a list of sorted int32 arrays of vocabulary ids, one per row; with
    margin 0 each holds exactly ``sample_select``'s token (a target that sits
    on an interval edge adds the member the edge belongs to).  Pinned by that
    identity and by a row with two equal weights at a CDF boundary, where both
    ids are candidates (tests/test_oracle.py).
    """
    f = np.asarray(f, dtype=np.float32)
    subset = np.asarray(subset, dtype=np.int64)
    M, n = f.shape
    tau = float(np.float32(temperature))
    tp = float(np.float32(top_p))
    out = []
    for m in range(M):
        x = f[m].astype(np.float64)
        e = np.exp((x - x.max()) / tau)
        p = e / e.sum()
        order = np.lexsort((subset, -p))
        cum = np.cumsum(p[order])
        if tp >= 1.0:
            k_lo = k_hi = n
        else:
            k_lo = min(int(np.searchsorted(cum, tp - margin, side="left")) + 1, n)
            k_hi = min(int(np.searchsorted(cum, tp + margin, side="left")) + 1, n)
        g = m if row_index is None else int(row_index[m])
        u = philox_uniform(seed, g % rows_per_session, g // rows_per_session)
        cand = set()
        for K in range(max(k_lo, 1), k_hi + 1):
            members = np.sort(order[:K])
            run = np.cumsum(p[members])
            target = u * run[-1]
            before = np.concatenate(([0.0], run[:-1]))
            # member i is drawn when before[i] <= target < run[i]
            hit = (before <= target + margin) & (run >= target - margin)
            if target + margin >= run[-1]:
                hit[-1] = True          # the fallback pick when rounding leaves none
            cand.update(subset[members[hit]].tolist())
        out.append(np.array(sorted(cand), dtype=np.int32))
    return out


# ---------------------------------------------------------------------------
# verification of the drafts (Section 5.5, Algorithm 1)
# ---------------------------------------------------------------------------


def accept_lengths(tokens, drafts, n_sessions, rows_per_session) -> np.ndarray:
    """Accepted draft-prefix length per session.

    Session s verifies rows s*R .. s*R+R-1 (R = k + 1).  Row r produces the
    token that draft r must equal; the session keeps the longest prefix of
    drafts that all match, a_s in [0, k].  Committed tokens are then drafts
    [0, a_s) followed by the token of row a_s (the correction, or the bonus
    token when every draft matched).
    """
    R = int(rows_per_session)
    k = R - 1
    tokens = np.asarray(tokens).reshape(n_sessions, R)
    out = np.zeros(n_sessions, dtype=np.int32)
    if k == 0:
        return out
    drafts = np.asarray(drafts).reshape(n_sessions, k)
    for s in range(n_sessions):
        a = 0
        while a < k and tokens[s, a] == drafts[s, a]:
            a += 1
        out[s] = a
    return out


# ---------------------------------------------------------------------------
# whole calls
# ---------------------------------------------------------------------------


def cloud_call(h_bits, d_end, subset, clip_c, w_cloud_bits=None, w_cloud_codes=None,
               w_cloud_scale=None, bias=None, rows=None, with_abs=False):
    """The cloud half of one decoding step (Algorithm 1, cloud partial):
    eq. 12 on S, then clip and int8 quantisation of each row."""
    z, absdot = cloud_partial_logits(h_bits, d_end, subset, w_cloud_bits, w_cloud_codes,
                                     w_cloud_scale, bias, rows=rows, with_abs=with_abs)
    out = clip_quantize(z, clip_c)
    out["z"] = z
    out["absdot"] = absdot
    return out


def endpoint_call(q, scale, h_bits, d_end, subset, w_end_bits, n_sessions, rows_per_session,
                  drafts=None, mode="greedy", temperature=1.0, top_p=1.0, seed=0,
                  with_abs=False):
    """The endpoint half of one decoding step: eq. 11 on S, dequantise + fuse
    + mask (eq. 13-14), select (eq. 15), then the accepted draft prefix."""
    z_e, absdot = endpoint_partial_logits(h_bits, d_end, subset, w_end_bits, with_abs=with_abs)
    f = fuse_masked(q, scale, z_e)
    out = {"z_end": z_e, "absdot": absdot, "f": f}
    if mode == "greedy":
        tok, pos, gap = greedy_select(f, subset)
        out.update(tokens=tok, pos=pos, gap=gap)
    elif mode == "sample":
        tok, info = sample_select(f, subset, temperature, top_p, seed, rows_per_session)
        out.update(tokens=tok, **info)
    else:
        raise ValueError(mode)
    out["accept"] = accept_lengths(out["tokens"], drafts, n_sessions, rows_per_session)
    return out
