"""Pins of the AES-GCM oracle (eq. 19): published known-answer values of
FIPS-197 and of the GCM specification, field identities, and agreement with
the system OpenSSL (libcrypto, called through ctypes) where it loads."""

import ctypes
import ctypes.util

import numpy as np
import pytest

from oracle import gcm

H = bytes.fromhex


# ---------------------------------------------------------------------------
# FIPS-197
# ---------------------------------------------------------------------------

def test_gf256_products_of_the_standard():
    # Section 4.2: {57} . {83} = {c1}; Section 4.2.1: {57} . {13} = {fe}
    assert gcm.gf256_mul(0x57, 0x83) == 0xC1
    assert gcm.gf256_mul(0x57, 0x13) == 0xFE


def test_sbox_values_and_permutation():
    s = gcm.SBOX
    assert s[0x00] == 0x63 and s[0x01] == 0x7C and s[0x53] == 0xED   # Section 5.1.1 example: {53} -> {ed}
    assert sorted(s.tolist()) == list(range(256))
    assert not np.any(s == np.arange(256))                             # no fixed points


def test_key_expansion_appendix_a1():
    rk = gcm.expand_key(H("2b7e151628aed2a6abf7158809cf4f3c"))
    assert rk.shape == (11, 16)
    assert rk[1, :4].tobytes() == H("a0fafe17")                        # w[4]
    assert rk[10, 12:].tobytes() == H("b6630ca6")                      # w[43]


@pytest.mark.parametrize("key,pt,ct", [
    ("2b7e151628aed2a6abf7158809cf4f3c", "3243f6a8885a308d313198a2e0370734",
     "3925841d02dc09fbdc118597196a0b32"),                              # Appendix B
    ("000102030405060708090a0b0c0d0e0f", "00112233445566778899aabbccddeeff",
     "69c4e0d86a7b0430d8cdb78070b4c55a"),                              # Appendix C.1
    ("000102030405060708090a0b0c0d0e0f101112131415161718191a1b1c1d1e1f",
     "00112233445566778899aabbccddeeff", "8ea2b7ca516745bfeafc49904b496089"),  # Appendix C.3
])
def test_cipher_known_answers(key, pt, ct):
    rk = gcm.expand_key(H(key))
    out = gcm.aes_encrypt_blocks(rk, np.frombuffer(H(pt), np.uint8).reshape(1, 16))
    assert out.tobytes() == H(ct)


# ---------------------------------------------------------------------------
# GCM
# ---------------------------------------------------------------------------

_P3 = ("d9313225f88406e5a55909c5aff5269a86a7a9531534f7da2e4c303d8a318a72"
       "1c3c0c95956809532fcf0e2449a6b525b16aedf5aa0de657ba637b391aafd255")
_C3 = ("42831ec2217774244b7221b784d0d49ce3aa212f2c02a4e035c17e2329aca12e"
       "21d514b25466931c7d8f6a5aac84aa051ba30b396a0aac973d58e091473f5985")


@pytest.mark.parametrize("key,iv,pt,aad,ct,tag", [
    # the specification's test cases 1-4 (AES-128)
    ("00" * 16, "00" * 12, "", "", "", "58e2fccefa7e3061367f1d57a4e7455a"),
    ("00" * 16, "00" * 12, "00" * 16, "", "0388dace60b6a392f328c2b971b2fe78",
     "ab6e47d42cec13bdf53a67b21257bddf"),
    ("feffe9928665731c6d6a8f9467308308", "cafebabefacedbaddecaf888", _P3, "", _C3,
     "4d5c2af327cd64a62cf35abd2ba6fab4"),
    ("feffe9928665731c6d6a8f9467308308", "cafebabefacedbaddecaf888", _P3[:120],
     "feedfacedeadbeeffeedfacedeadbeefabaddad2", _C3[:120], "5bc94fbc3221a5db94fae95ae7121a47"),
])
def test_gcm_known_answers(key, iv, pt, aad, ct, tag):
    c, t = gcm.gcm_encrypt(H(key), H(iv), H(pt), H(aad))
    assert c == H(ct) and t == H(tag)
    p, ok = gcm.gcm_decrypt(H(key), H(iv), c, t, H(aad))
    assert ok and p == H(pt)
    bad = bytes([t[0] ^ 1]) + t[1:]
    assert not gcm.gcm_decrypt(H(key), H(iv), c, bad, H(aad))[1]


def test_gf128_field_identities():
    rng = np.random.default_rng(5)
    one = 1 << 127                        # the block 80 00 .. 00 is the polynomial 1
    xs = [int.from_bytes(rng.bytes(16), "big") for _ in range(6)]
    for a, b, c in zip(xs[0::3], xs[1::3], xs[2::3]):
        assert gcm.gf128_mul(a, one) == a
        assert gcm.gf128_mul(a, b) == gcm.gf128_mul(b, a)
        assert gcm.gf128_mul(a, b ^ c) == gcm.gf128_mul(a, b) ^ gcm.gf128_mul(a, c)
        assert gcm.gf128_mul(gcm.gf128_mul(a, b), c) == gcm.gf128_mul(a, gcm.gf128_mul(b, c))


# ---------------------------------------------------------------------------
# agreement with OpenSSL (system libcrypto), if it can be loaded
# ---------------------------------------------------------------------------

def _libcrypto():
    name = ctypes.util.find_library("crypto")
    if not name:
        return None
    try:
        lib = ctypes.CDLL(name)
        lib.EVP_CIPHER_CTX_new.restype = ctypes.c_void_p
        lib.EVP_aes_128_gcm.restype = ctypes.c_void_p
        lib.EVP_aes_256_gcm.restype = ctypes.c_void_p
        return lib
    except (OSError, AttributeError):
        return None


def _openssl_gcm(lib, key, iv, pt, aad):
    EVP_CTRL_GCM_GET_TAG = 0x10
    ctx = ctypes.c_void_p(lib.EVP_CIPHER_CTX_new())
    cipher = ctypes.c_void_p(lib.EVP_aes_128_gcm() if len(key) == 16 else lib.EVP_aes_256_gcm())
    assert lib.EVP_EncryptInit_ex(ctx, cipher, None, key, iv) == 1
    n = ctypes.c_int(0)
    if aad:
        assert lib.EVP_EncryptUpdate(ctx, None, ctypes.byref(n), aad, len(aad)) == 1
    out = ctypes.create_string_buffer(len(pt) + 16)
    if pt:
        assert lib.EVP_EncryptUpdate(ctx, out, ctypes.byref(n), pt, len(pt)) == 1
    fin = ctypes.create_string_buffer(16)
    assert lib.EVP_EncryptFinal_ex(ctx, fin, ctypes.byref(n)) == 1
    tag = ctypes.create_string_buffer(16)
    assert lib.EVP_CIPHER_CTX_ctrl(ctx, EVP_CTRL_GCM_GET_TAG, 16, tag) == 1
    lib.EVP_CIPHER_CTX_free(ctx)
    return out.raw[:len(pt)], tag.raw


@pytest.mark.parametrize("klen", [16, 32])
@pytest.mark.parametrize("plen,alen", [(0, 0), (1, 3), (15, 0), (16, 16), (17, 20), (100, 45),
                                      (1000, 7), (4099, 64)])
def test_gcm_matches_openssl(klen, plen, alen):
    lib = _libcrypto()
    if lib is None:
        pytest.skip("libcrypto not loadable")
    rng = np.random.default_rng(plen * 31 + alen + klen)
    key, iv, pt, aad = rng.bytes(klen), rng.bytes(12), rng.bytes(plen), rng.bytes(alen)
    assert gcm.gcm_encrypt(key, iv, pt, aad) == _openssl_gcm(lib, key, iv, pt, aad)


def test_seal_rows_is_per_row_gcm():
    rng = np.random.default_rng(9)
    key = rng.bytes(16)
    rows = rng.integers(0, 256, (3, 40), dtype=np.uint8)
    ivs = rng.integers(0, 256, (3, 12), dtype=np.uint8)
    aads = rng.integers(0, 256, (3, 5), dtype=np.uint8)
    ct, tags = gcm.seal_rows(key, rows, ivs, aads)
    for m in range(3):
        c, t = gcm.gcm_encrypt(key, ivs[m].tobytes(), rows[m].tobytes(), aads[m].tobytes())
        assert ct[m].tobytes() == c and tags[m].tobytes() == t
