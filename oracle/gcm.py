"""AES and Galois/Counter Mode for the payload seal of eq. 19.

TEST INFRASTRUCTURE ONLY (see the package docstring): the HIP library never
calls this module, and they share no table or constant generator.

Eq. 19 encrypts each quantised payload with AES-GCM under a key K and a nonce
IV, authenticating session, block and cache metadata as associated data.
This is a plain restatement of the two standards the paper names:

  * AES (FIPS-197): the S-box is computed from its definition (the
    multiplicative inverse in GF(2^8) modulo x^8 + x^4 + x^3 + x + 1,
    followed by the affine map with constant 0x63), then key expansion and
    the cipher (SubBytes, ShiftRows, MixColumns, AddRoundKey) for 128- and
    256-bit keys, evaluated on many blocks at once with NumPy.
  * GCM (NIST SP 800-38D) with a 96-bit IV: H = E_K(0^128),
    J0 = IV || 0^31 || 1, C = GCTR(inc32(J0), P), the tag
    E_K(J0) xor GHASH_H(A || pad || C || pad || [len A]_64 || [len C]_64),
    with the bit-serial multiplication in GF(2^128) of the standard
    (R = 11100001 || 0^120, the leftmost bit the lowest power).

Pinned by the published known-answer values of both standards (FIPS-197
appendix vectors, the GCM specification's test cases) and by the system
OpenSSL where it can be loaded.
"""

from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------------------
# GF(2^8) and the S-box (FIPS-197 Section 4 and 5.1.1)
# ---------------------------------------------------------------------------


def gf256_mul(a: int, b: int) -> int:
    """Product in GF(2^8) modulo x^8 + x^4 + x^3 + x + 1 (shift and add)."""
    r = 0
    while b:
        if b & 1:
            r ^= a
        a <<= 1
        if a & 0x100:
            a ^= 0x11B
        b >>= 1
    return r


def _gf256_inverse(a: int) -> int:
    """a^254 = a^-1 for a != 0 (the group of units has order 255); 0 -> 0."""
    if a == 0:
        return 0
    r, p, e = 1, a, 254
    while e:
        if e & 1:
            r = gf256_mul(r, p)
        p = gf256_mul(p, p)
        e >>= 1
    return r


def _rotl8(x: int, k: int) -> int:
    return ((x << k) | (x >> (8 - k))) & 0xFF


def make_sbox() -> np.ndarray:
    """S(x) = affine(inverse(x)): b ^ rotl(b,1) ^ rotl(b,2) ^ rotl(b,3) ^
    rotl(b,4) ^ 0x63, which is FIPS-197 eq. 5.1 written with rotations."""
    s = np.zeros(256, dtype=np.uint8)
    for x in range(256):
        b = _gf256_inverse(x)
        s[x] = b ^ _rotl8(b, 1) ^ _rotl8(b, 2) ^ _rotl8(b, 3) ^ _rotl8(b, 4) ^ 0x63
    return s


SBOX = make_sbox()
_MUL2 = np.array([gf256_mul(x, 2) for x in range(256)], dtype=np.uint8)
_MUL3 = np.array([gf256_mul(x, 3) for x in range(256)], dtype=np.uint8)


# ---------------------------------------------------------------------------
# key expansion and the cipher (FIPS-197 Sections 5.1 and 5.2)
# ---------------------------------------------------------------------------


def expand_key(key: bytes) -> np.ndarray:
    """Round keys as uint8 [Nr + 1, 16] (column-major state order) for a
    16- or 32-byte key (Nk = 4, Nr = 10 or Nk = 8, Nr = 14)."""
    key = bytes(key)
    if len(key) not in (16, 32):
        raise ValueError("AES key must be 16 or 32 bytes")
    nk = len(key) // 4
    nr = nk + 6
    w = [list(key[4 * i:4 * i + 4]) for i in range(nk)]
    rcon = 1
    for i in range(nk, 4 * (nr + 1)):
        t = list(w[i - 1])
        if i % nk == 0:
            t = t[1:] + t[:1]                       # RotWord
            t = [int(SBOX[b]) for b in t]           # SubWord
            t[0] ^= rcon
            rcon = gf256_mul(rcon, 2)
        elif nk > 6 and i % nk == 4:
            t = [int(SBOX[b]) for b in t]
        w.append([w[i - nk][j] ^ t[j] for j in range(4)])
    rk = np.array(w, dtype=np.uint8).reshape(nr + 1, 16)
    return rk


def aes_encrypt_blocks(rk: np.ndarray, blocks: np.ndarray) -> np.ndarray:
    """The cipher on uint8 [B, 16] blocks.  Byte i of a block is state
    element (row i % 4, column i // 4)."""
    nr = rk.shape[0] - 1
    s = np.asarray(blocks, dtype=np.uint8).reshape(-1, 4, 4).copy()   # [B, column, row]
    s ^= rk[0].reshape(4, 4)
    for rnd in range(1, nr + 1):
        s = SBOX[s]                                                     # SubBytes
        t = np.empty_like(s)
        for r in range(4):                                              # ShiftRows: row r left by r
            t[:, :, r] = np.roll(s[:, :, r], -r, axis=1)
        s = t
        if rnd != nr:                                                   # MixColumns
            a0, a1, a2, a3 = (s[:, :, r] for r in range(4))
            s = np.stack([_MUL2[a0] ^ _MUL3[a1] ^ a2 ^ a3,
                          a0 ^ _MUL2[a1] ^ _MUL3[a2] ^ a3,
                          a0 ^ a1 ^ _MUL2[a2] ^ _MUL3[a3],
                          _MUL3[a0] ^ a1 ^ a2 ^ _MUL2[a3]], axis=2)
        s ^= rk[rnd].reshape(4, 4)
    return s.reshape(-1, 16)


# ---------------------------------------------------------------------------
# GCM (NIST SP 800-38D Sections 6 and 7), 96-bit IV
# ---------------------------------------------------------------------------

_R = 0xE1 << 120


def gf128_mul(x: int, y: int) -> int:
    """X . Y in GF(2^128), blocks as integers read big-endian (the leftmost
    bit of a block is the integer's bit 127): the standard's Algorithm 1."""
    z, v = 0, y
    for i in range(127, -1, -1):
        if (x >> i) & 1:
            z ^= v
        v = (v >> 1) ^ _R if v & 1 else v >> 1
    return z


def ghash(h: int, data: bytes) -> int:
    """GHASH_H of a whole number of 16-byte blocks."""
    assert len(data) % 16 == 0
    y = 0
    for i in range(0, len(data), 16):
        y = gf128_mul(y ^ int.from_bytes(data[i:i + 16], "big"), h)
    return y


def _counter_blocks(iv: bytes, first: int, count: int) -> np.ndarray:
    """IV || [first + i mod 2^32]_32 for i < count (inc32 from first)."""
    blocks = np.zeros((count, 16), dtype=np.uint8)
    blocks[:, :12] = np.frombuffer(bytes(iv), dtype=np.uint8)
    ctr = (first + np.arange(count, dtype=np.uint64)) & 0xFFFFFFFF
    for k in range(4):
        blocks[:, 12 + k] = (ctr >> np.uint64(8 * (3 - k))) & 0xFF
    return blocks


def _pad16(b: bytes) -> bytes:
    return b + bytes(-len(b) % 16)


def _tag(rk, h, iv, aad, ct):
    s = ghash(h, _pad16(aad) + _pad16(ct) + (8 * len(aad)).to_bytes(8, "big")
              + (8 * len(ct)).to_bytes(8, "big"))
    e0 = aes_encrypt_blocks(rk, _counter_blocks(iv, 1, 1))[0]
    return (int.from_bytes(e0.tobytes(), "big") ^ s).to_bytes(16, "big")


def gcm_encrypt(key: bytes, iv: bytes, plaintext: bytes, aad: bytes = b""):
    """Authenticated encryption: returns (ciphertext, 16-byte tag)."""
    if len(iv) != 12:
        raise ValueError("this oracle takes 96-bit IVs")
    rk = expand_key(key)
    h = int.from_bytes(aes_encrypt_blocks(rk, np.zeros((1, 16), np.uint8))[0].tobytes(), "big")
    pt = bytes(plaintext)
    n = -(-len(pt) // 16)
    ks = aes_encrypt_blocks(rk, _counter_blocks(iv, 2, n)).tobytes()[:len(pt)] if n else b""
    ct = bytes(a ^ b for a, b in zip(pt, ks))
    return ct, _tag(rk, h, iv, bytes(aad), ct)


def gcm_decrypt(key: bytes, iv: bytes, ciphertext: bytes, tag: bytes, aad: bytes = b""):
    """Authenticated decryption: returns (plaintext, tag_ok)."""
    rk = expand_key(key)
    h = int.from_bytes(aes_encrypt_blocks(rk, np.zeros((1, 16), np.uint8))[0].tobytes(), "big")
    ct = bytes(ciphertext)
    n = -(-len(ct) // 16)
    ks = aes_encrypt_blocks(rk, _counter_blocks(iv, 2, n)).tobytes()[:len(ct)] if n else b""
    pt = bytes(a ^ b for a, b in zip(ct, ks))
    return pt, _tag(rk, h, iv, bytes(aad), ct) == bytes(tag)


def seal_rows(key: bytes, rows: np.ndarray, ivs: np.ndarray, aads: np.ndarray):
    """Eq. 19 on a batch of payload rows, each its own message: row m is
    encrypted under IV ivs[m] (12 bytes) with associated data aads[m].
    Returns (ciphertext uint8 [M, L], tags uint8 [M, 16])."""
    rows = np.asarray(rows, dtype=np.uint8)
    ct = np.zeros_like(rows)
    tags = np.zeros((rows.shape[0], 16), np.uint8)
    for m in range(rows.shape[0]):
        c, t = gcm_encrypt(key, bytes(ivs[m]), rows[m].tobytes(), bytes(aads[m]))
        ct[m] = np.frombuffer(c, np.uint8)
        tags[m] = np.frombuffer(t, np.uint8)
    return ct, tags
