// AES-GCM seal and open of payload rows (eq. 19: the quantised payload is
// encrypted with AES-GCM under a key K and a nonce IV, with session, block
// and cache metadata as associated data).  AES per FIPS-197, GCM per NIST
// SP 800-38D with 96-bit IVs; every row is its own message.
//
// Key set-up (host, once per key): the S-box from its definition (inverse
// in GF(2^8) by discrete logarithms to the generator 3, then the affine map
// bit by bit), one 256-entry table T0[x] = (2S(x), S(x), S(x), 3S(x)) whose
// byte rotations give the other three column tables, the round keys, the
// hash key H = E_K(0^128) and the powers H^1 .. H^kGcmMaxPow.
//
// GHASH of a message with a AAD blocks, n ciphertext blocks and the length
// block is S = sum_k X_k H^(m-k+1), m = a + n + 1, so with the powers in a
// table every block's term is independent: ciphertext block j (0-based)
// contributes C_j H^(n+1-j).  k_gcm_blocks runs one thread per 16-byte
// block (counter-mode keystream from inc32 counters 2, 3, ... and the
// block's GHASH term) and XOR-reduces the terms of its 256 blocks;
// k_gcm_finish adds the partial sums, the AAD and length terms and forms
// (seal) or checks (open) the tag E_K(J0) xor S.  XOR is exact and
// associative, so the result does not depend on the reduction order.
#include <cstring>
#include <vector>

#include "sph_internal.h"

namespace sph {

namespace {

// ---------------------------------------------------------------------------
// host: S-box, tables, key schedule, powers of H
// ---------------------------------------------------------------------------

uint8_t xtime(uint8_t b) { return (uint8_t)((b << 1) ^ ((b & 0x80) ? 0x1B : 0x00)); }

void build_sbox(uint8_t sbox[256]) {
  // 3 generates the multiplicative group of GF(2^8): log / antilog tables
  uint8_t alog[255];
  int lg[256] = {0};
  uint8_t x = 1;
  for (int i = 0; i < 255; ++i) {
    alog[i] = x;
    lg[x] = i;
    x = (uint8_t)(x ^ xtime(x));  // x * 3
  }
  for (int a = 0; a < 256; ++a) {
    const uint8_t inv = a == 0 ? 0 : alog[(255 - lg[a]) % 255];
    // affine map: bit i of the result = b_i ^ b_(i+4) ^ b_(i+5) ^ b_(i+6) ^ b_(i+7) ^ c_i (indices mod 8)
    uint8_t r = 0;
    for (int i = 0; i < 8; ++i) {
      const int bit = ((inv >> i) ^ (inv >> ((i + 4) & 7)) ^ (inv >> ((i + 5) & 7)) ^
                       (inv >> ((i + 6) & 7)) ^ (inv >> ((i + 7) & 7)) ^ (0x63 >> i)) & 1;
      r = (uint8_t)(r | (bit << i));
    }
    sbox[a] = r;
  }
}

uint32_t rotr32(uint32_t v, int k) { return (v >> k) | (v << (32 - k)); }

}  // namespace

// words are big-endian: byte 0 of a column (row 0) is the most significant
__host__ __device__ __forceinline__ uint32_t gcm_rotr(uint32_t v, int k) {
  return (v >> k) | (v << (32 - k));
}

// One AES block: in/out as four big-endian column words.  te: the T0 table,
// sb: the S-box, rk: 4 (nr + 1) round-key words.
template <class TE, class SB, class RK>
__host__ __device__ __forceinline__ void aes_block(TE te, SB sb, RK rk, int nr, const uint32_t in[4],
                                                   uint32_t out[4]) {
  uint32_t s0 = in[0] ^ rk[0], s1 = in[1] ^ rk[1], s2 = in[2] ^ rk[2], s3 = in[3] ^ rk[3];
#pragma unroll
  for (int r = 1; r < nr; ++r) {
    // column c of the next state: T0[row 0 of column c] ^ T1[row 1 of c+1]
    // ^ T2[row 2 of c+2] ^ T3[row 3 of c+3] ^ round key (ShiftRows folded in)
    const uint32_t t0 = te[s0 >> 24] ^ gcm_rotr(te[(s1 >> 16) & 255], 8) ^
                        gcm_rotr(te[(s2 >> 8) & 255], 16) ^ gcm_rotr(te[s3 & 255], 24) ^ rk[4 * r];
    const uint32_t t1 = te[s1 >> 24] ^ gcm_rotr(te[(s2 >> 16) & 255], 8) ^
                        gcm_rotr(te[(s3 >> 8) & 255], 16) ^ gcm_rotr(te[s0 & 255], 24) ^ rk[4 * r + 1];
    const uint32_t t2 = te[s2 >> 24] ^ gcm_rotr(te[(s3 >> 16) & 255], 8) ^
                        gcm_rotr(te[(s0 >> 8) & 255], 16) ^ gcm_rotr(te[s1 & 255], 24) ^ rk[4 * r + 2];
    const uint32_t t3 = te[s3 >> 24] ^ gcm_rotr(te[(s0 >> 16) & 255], 8) ^
                        gcm_rotr(te[(s1 >> 8) & 255], 16) ^ gcm_rotr(te[s2 & 255], 24) ^ rk[4 * r + 3];
    s0 = t0; s1 = t1; s2 = t2; s3 = t3;
  }
  // last round: SubBytes and ShiftRows only
  auto last = [&](uint32_t a, uint32_t b, uint32_t c, uint32_t d, uint32_t k) {
    return (((uint32_t)sb[a >> 24]) << 24 | ((uint32_t)sb[(b >> 16) & 255]) << 16 |
            ((uint32_t)sb[(c >> 8) & 255]) << 8 | (uint32_t)sb[d & 255]) ^ k;
  };
  out[0] = last(s0, s1, s2, s3, rk[4 * nr]);
  out[1] = last(s1, s2, s3, s0, rk[4 * nr + 1]);
  out[2] = last(s2, s3, s0, s1, rk[4 * nr + 2]);
  out[3] = last(s3, s0, s1, s2, rk[4 * nr + 3]);
}

// z = x . y in GF(2^128) (the standard's bit-serial product: bit i of x
// from the left selects V_i, V_(i+1) = V_i >> 1 reduced by R = 0xE1 || 0^120).
__host__ __device__ __forceinline__ void gf128_mul(const uint32_t x[4], const uint32_t y[4],
                                                   uint32_t z[4]) {
  uint32_t v0 = y[0], v1 = y[1], v2 = y[2], v3 = y[3];
  uint32_t z0 = 0, z1 = 0, z2 = 0, z3 = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t xw = x[w];
#pragma unroll 8
    for (int b = 31; b >= 0; --b) {
      const uint32_t m = 0u - ((xw >> b) & 1u);
      z0 ^= v0 & m; z1 ^= v1 & m; z2 ^= v2 & m; z3 ^= v3 & m;
      const uint32_t lsb = 0u - (v3 & 1u);
      v3 = (v3 >> 1) | (v2 << 31);
      v2 = (v2 >> 1) | (v1 << 31);
      v1 = (v1 >> 1) | (v0 << 31);
      v0 = (v0 >> 1) ^ (0xE1000000u & lsb);
    }
  }
  z[0] = z0; z[1] = z1; z[2] = z2; z[3] = z3;
}

bool gcm_key_setup(const uint8_t* key, int key_bytes, std::vector<uint8_t>& dev_image, int& nr) {
  if (key_bytes != 16 && key_bytes != 32) return false;
  uint8_t sbox[256];
  build_sbox(sbox);
  uint32_t te[256];
  for (int x = 0; x < 256; ++x) {
    const uint8_t s = sbox[x], s2 = xtime(s), s3 = (uint8_t)(s2 ^ s);
    te[x] = ((uint32_t)s2 << 24) | ((uint32_t)s << 16) | ((uint32_t)s << 8) | s3;
  }
  const int nk = key_bytes / 4;
  nr = nk + 6;
  uint32_t w[60];
  for (int i = 0; i < nk; ++i)
    w[i] = ((uint32_t)key[4 * i] << 24) | ((uint32_t)key[4 * i + 1] << 16) |
           ((uint32_t)key[4 * i + 2] << 8) | key[4 * i + 3];
  uint8_t rc = 1;
  auto subword = [&](uint32_t v) {
    return ((uint32_t)sbox[v >> 24] << 24) | ((uint32_t)sbox[(v >> 16) & 255] << 16) |
           ((uint32_t)sbox[(v >> 8) & 255] << 8) | sbox[v & 255];
  };
  for (int i = nk; i < 4 * (nr + 1); ++i) {
    uint32_t t = w[i - 1];
    if (i % nk == 0) {
      t = subword(rotr32(t, 24)) ^ ((uint32_t)rc << 24);  // RotWord is a left byte rotation
      rc = xtime(rc);
    } else if (nk > 6 && i % nk == 4) {
      t = subword(t);
    }
    w[i] = w[i - nk] ^ t;
  }
  // device image: te | sbox | round keys | powers of H
  dev_image.assign(kGcmImageBytes, 0);
  std::memcpy(dev_image.data(), te, sizeof(te));
  std::memcpy(dev_image.data() + 1024, sbox, 256);
  std::memcpy(dev_image.data() + kGcmRkOffset, w, sizeof(uint32_t) * 4 * (nr + 1));
  const uint32_t zero[4] = {0, 0, 0, 0};
  uint32_t h[4];
  aes_block(te, sbox, w, nr, zero, h);
  uint32_t* pw = reinterpret_cast<uint32_t*>(dev_image.data() + kGcmPowOffset);  // pw[4e .. 4e+3] = H^e
  std::memcpy(pw + 4, h, 16);
  for (int e = 2; e <= kGcmMaxPow; ++e) gf128_mul(pw + 4 * (e - 1), h, pw + 4 * e);
  // nibble tables of the product by G = H^kGcmStride (the product is linear
  // in its first factor, so Y.G is the xor of the entries of Y's nibbles)
  uint32_t* tab = reinterpret_cast<uint32_t*>(dev_image.data() + kGcmTabOffset);
  for (int p = 0; p < 32; ++p)
    for (int v = 0; v < 16; ++v) {
      uint32_t x[4] = {0u, 0u, 0u, 0u};
      x[p >> 3] = (uint32_t)v << (28 - 4 * (p & 7));
      gf128_mul(x, pw + 4 * kGcmStride, tab + 4 * (16 * p + v));
    }
  return true;
}

// ---------------------------------------------------------------------------
// device
// ---------------------------------------------------------------------------

__device__ __forceinline__ void pack_be_words(const uint8_t b[16], uint32_t w[4]) {
#pragma unroll
  for (int k = 0; k < 4; ++k)
    w[k] = ((uint32_t)b[4 * k] << 24) | ((uint32_t)b[4 * k + 1] << 16) | ((uint32_t)b[4 * k + 2] << 8) |
           b[4 * k + 3];
}

__device__ __forceinline__ void load_be_words(const uint8_t* p, int valid, uint32_t w[4]) {
  uint8_t b[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) b[i] = i < valid ? p[i] : 0;
  pack_be_words(b, w);
}

// Segment of a message row that holds message byte p (p < L): the last
// segment starting at or before p, so empty segments are passed over.
__device__ __forceinline__ int seg_of(const GcmSegs& g, int64_t p, int64_t& start) {
  int s = 0;
  start = 0;
#pragma unroll
  for (int k = 0; k < kGcmMaxSegs - 1; ++k)
    if (k + 1 < g.nseg && p >= g.end[k]) {
      s = k + 1;
      start = g.end[k];
    }
  return s;
}

template <typename T>
__device__ __forceinline__ T* seg_ptr(T* const (&base)[kGcmMaxSegs], const int64_t (&ld)[kGcmMaxSegs],
                                      int s, int64_t row, int64_t off) {
  T* b = base[0];
  int64_t l = ld[0];
#pragma unroll
  for (int k = 1; k < kGcmMaxSegs; ++k)
    if (s == k) {
      b = base[k];
      l = ld[k];
    }
  return b + row * l + off;
}

// The T0 table sits in LDS as kTeSlices copies, entry x of copy c at word
// x * kTeSlices + c, and lane l reads copy l mod kTeSlices: lanes that share
// a bank are then the lanes l, l + 16, l + 32, l + 48, where one table would
// let any two of the 64 lanes collide.  The S-box is byte 1 of T0
// (T0[x] = (2S(x), S(x), S(x), 3S(x))).
constexpr int kTeSlices = 16;

struct GcmShared {
  __attribute__((aligned(16))) uint32_t te[256 * kTeSlices];
  uint32_t rk[60];
  uint32_t red[4][4];
};

struct TeSlice {
  const uint32_t* t;  // the lane's copy
  __device__ __forceinline__ uint32_t operator[](uint32_t x) const { return t[x * kTeSlices]; }
};
struct SboxSlice {
  const uint32_t* t;
  __device__ __forceinline__ uint8_t operator[](uint32_t x) const {
    return (uint8_t)(t[x * kTeSlices] >> 16);
  }
};

__device__ __forceinline__ void stage_key(GcmShared& sh, const uint8_t* key_dev, int nr) {
  const int tid = threadIdx.x;
  const uint32_t* te = reinterpret_cast<const uint32_t*>(key_dev);
  // one global load per entry, its copies written as 16-byte stores
  for (int x = tid; x < 256; x += blockDim.x) {
    const uint32_t v = te[x];
#pragma unroll
    for (int q = 0; q < kTeSlices / 4; ++q)
      *reinterpret_cast<uint4*>(&sh.te[x * kTeSlices + 4 * q]) = make_uint4(v, v, v, v);
  }
  if (tid < 4 * (nr + 1)) sh.rk[tid] = reinterpret_cast<const uint32_t*>(key_dev + kGcmRkOffset)[tid];
  __syncthreads();
}

__device__ __forceinline__ void aes_block_lds(const GcmShared& sh, int nr, const uint32_t in[4],
                                              uint32_t out[4]) {
  const uint32_t* t = sh.te + (threadIdx.x & (kTeSlices - 1));
  aes_block(TeSlice{t}, SboxSlice{t}, sh.rk, nr, in, out);
}

// Y . G from the nibble tables in LDS: 32 independent lookups, no shifts.
__device__ __forceinline__ void mul_by_g(uint32_t y[4], const uint4* __restrict__ tab) {
  uint32_t r0 = 0u, r1 = 0u, r2 = 0u, r3 = 0u;
#pragma unroll
  for (int p = 0; p < 32; ++p) {
    const uint32_t v = (y[p >> 3] >> (28 - 4 * (p & 7))) & 15u;
    const uint4 e = tab[16 * p + v];
    r0 ^= e.x;
    r1 ^= e.y;
    r2 ^= e.z;
    r3 ^= e.w;
  }
  y[0] = r0;
  y[1] = r1;
  y[2] = r2;
  y[3] = r3;
}

// Counter-mode output of data block j of a row and its GHASH input (the
// ciphertext, zero past the message).
template <bool OPEN, int NR>
__device__ __forceinline__ void gcm_data_block(const GcmShared& sh, const GcmSegs& segs,
                                               int64_t L, const uint32_t ivw[3], int64_t row, int j,
                                               uint32_t c[4]) {
  uint32_t ctr[4] = {ivw[0], ivw[1], ivw[2], (uint32_t)(2 + j)};  // inc32 from J0 + 1
  uint32_t ks[4];
  aes_block_lds(sh, NR, ctr, ks);
  const int64_t p0 = (int64_t)j * 16;
  const int valid = (int)min<int64_t>(16, L - p0);
  int64_t st;
  const int s0 = seg_of(segs, p0, st);
  int64_t e0 = segs.end[0];
#pragma unroll
  for (int k = 1; k < kGcmMaxSegs; ++k)
    if (s0 == k) e0 = segs.end[k];
  // a block inside one segment takes the plain path; one that straddles a
  // segment boundary maps every byte on its own
  const bool whole = p0 + valid <= e0;
  uint32_t x[4], y[4];
  if (whole) {
    const uint8_t* src = seg_ptr(segs.in, segs.ld_in, s0, row, p0 - st);
    if (valid == 16 && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
      const uint4 v = *reinterpret_cast<const uint4*>(src);
      x[0] = __builtin_bswap32(v.x);
      x[1] = __builtin_bswap32(v.y);
      x[2] = __builtin_bswap32(v.z);
      x[3] = __builtin_bswap32(v.w);
    } else {
      load_be_words(src, valid, x);
    }
  } else {
    uint8_t b[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      b[i] = 0;
      if (i < valid) {
        int64_t sti;
        const int si = seg_of(segs, p0 + i, sti);
        b[i] = *seg_ptr(segs.in, segs.ld_in, si, row, p0 + i - sti);
      }
    }
    pack_be_words(b, x);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) y[k] = x[k] ^ ks[k];
  if (whole) {
    uint8_t* dst = seg_ptr(segs.out, segs.ld_out, s0, row, p0 - st);
    if (valid == 16 && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
      *reinterpret_cast<uint4*>(dst) = make_uint4(__builtin_bswap32(y[0]), __builtin_bswap32(y[1]),
                                                  __builtin_bswap32(y[2]), __builtin_bswap32(y[3]));
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (i < valid) dst[i] = (uint8_t)(y[i >> 2] >> (24 - 8 * (i & 3)));
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < valid) {
        int64_t sti;
        const int si = seg_of(segs, p0 + i, sti);
        *seg_ptr(segs.out, segs.ld_out, si, row, p0 + i - sti) = (uint8_t)(y[i >> 2] >> (24 - 8 * (i & 3)));
      }
  }
  // the GHASH input is the ciphertext: the output when sealing, the input
  // when opening
#pragma unroll
  for (int k = 0; k < 4; ++k) c[k] = OPEN ? x[k] : y[k];
  if (!OPEN && valid < 16) {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i >= valid) c[i >> 2] &= ~(0xFFu << (24 - 8 * (i & 3)));
  }
}

// GHASH of a message of na AAD blocks and n data blocks is the sum of the
// m = na + n + 1 terms X_k . H^(m+1-k) (k = 1..m, X_m the length block), and
// the tag is that sum xor E_K(J0).  Every term is independent given the
// powers of H.  Workgroup q of a row (grid: parts x rows) covers data blocks
// [q*S*chain, (q+1)*S*chain) with S = kGcmStride threads; thread t takes the
// blocks j_i = q*S*chain + t + S*i (i < chain, j_i < n), produces their
// output, and folds their terms by Horner's rule in G = H^S:
//   sum_i C_{j_i} . H^(n+1-j_i) = H^(n+1-j_last) . (...(C_{j_0} . G + C_{j_1}) . G ...)
// so each block costs one table product and each thread one bit-serial
// product by a power of H.  The last na + 2 threads of workgroup xpart
// (threads without a data block where threads take one block each) add the
// remaining terms: AAD block i (A_i . H^(m-i)), the length block times H,
// and E_K(J0).  Each workgroup xor-reduces its terms into one 16-byte
// partial of the row.
// NR: 10 rounds (AES-128) or 14 (AES-256), fixed so that the rounds unroll
template <bool OPEN, int NR>
__global__ __launch_bounds__(256) void k_gcm_blocks(const uint8_t* __restrict__ key_dev,
                                                    const GcmSegs segs, int64_t L, int n, int chain,
                                                    int xpart, const uint8_t* __restrict__ iv,
                                                    const uint8_t* __restrict__ aad, int64_t ld_aad,
                                                    int la, uint32_t* __restrict__ partial, int nparts) {
  __shared__ GcmShared sh;
  __shared__ uint4 tab[32 * 16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (chain > 1) {
    const uint4* src = reinterpret_cast<const uint4*>(key_dev + kGcmTabOffset);
    tab[tid] = src[tid];
    tab[tid + 256] = src[tid + 256];
  }
  stage_key(sh, key_dev, NR);  // ends with a barrier
  const int64_t row = blockIdx.y;
  const uint32_t* pw = reinterpret_cast<const uint32_t*>(key_dev + kGcmPowOffset);
  uint32_t ivw[4];
  load_be_words(iv + row * 12, 12, ivw);
  uint32_t t[4] = {0u, 0u, 0u, 0u};
  // data blocks
  {
    const int j0 = blockIdx.x * kGcmStride * chain + tid;
    uint32_t y[4] = {0u, 0u, 0u, 0u};
    int jl = -1;
    for (int i = 0; i < chain; ++i) {
      const int j = j0 + kGcmStride * i;
      if (j >= n) break;
      uint32_t c[4];
      gcm_data_block<OPEN, NR>(sh, segs, L, ivw, row, j, c);
      if (i > 0) mul_by_g(y, tab);
#pragma unroll
      for (int k = 0; k < 4; ++k) y[k] ^= c[k];
      jl = j;
    }
    if (jl >= 0) {
      const uint32_t* hp = pw + 4 * (n + 1 - jl);
      const uint32_t h4[4] = {hp[0], hp[1], hp[2], hp[3]};
      gf128_mul(y, h4, t);
    }
  }
  // AAD, length and E_K(J0) terms
  const int na = (la + 15) / 16;
  const int u = tid - (kGcmStride - (na + 2));
  if ((int)blockIdx.x == xpart && u >= 0) {
    const int m = na + n + 1;
    uint32_t c[4], r[4];
    if (u == na + 1) {
      const uint32_t j0b[4] = {ivw[0], ivw[1], ivw[2], 1u};
      aes_block_lds(sh, NR, j0b, r);
    } else {
      int e;
      if (u < na) {
        load_be_words(aad + row * ld_aad + (int64_t)u * 16, min(16, la - 16 * u), c);
        e = m - u;
      } else {
        const uint64_t abits = (uint64_t)la * 8, cbits = (uint64_t)L * 8;
        c[0] = (uint32_t)(abits >> 32);
        c[1] = (uint32_t)abits;
        c[2] = (uint32_t)(cbits >> 32);
        c[3] = (uint32_t)cbits;
        e = 1;
      }
      const uint32_t h4[4] = {pw[4 * e], pw[4 * e + 1], pw[4 * e + 2], pw[4 * e + 3]};
      gf128_mul(c, h4, r);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) t[k] ^= r[k];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) t[k] ^= __shfl_xor(t[k], o, 64);
    if (lane == 0) sh.red[wave][k] = t[k];
  }
  __syncthreads();
  if (tid < 4)
    partial[(row * nparts + blockIdx.x) * 4 + tid] = sh.red[0][tid] ^ sh.red[1][tid] ^ sh.red[2][tid] ^ sh.red[3][tid];
}

// One thread per row: the xor of the row's partials is its tag; write it
// (seal) or compare it with the given one in constant time (open).
template <bool OPEN>
__global__ __launch_bounds__(256) void k_gcm_finish(int rows, const uint32_t* __restrict__ partial,
                                                    int nparts, uint8_t* __restrict__ tag,
                                                    int32_t* __restrict__ ok) {
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (row >= rows) return;
  uint32_t s[4] = {0u, 0u, 0u, 0u};
  for (int p = 0; p < nparts; ++p)
#pragma unroll
    for (int k = 0; k < 4; ++k) s[k] ^= partial[(row * nparts + p) * 4 + k];
  uint8_t* tg = tag + row * 16;
  if (OPEN) {
    uint32_t diff = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) diff |= (uint32_t)((uint8_t)(s[i >> 2] >> (24 - 8 * (i & 3))) ^ tg[i]);
    ok[row] = diff == 0 ? 1 : 0;
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) tg[i] = (uint8_t)(s[i >> 2] >> (24 - 8 * (i & 3)));
  }
}

hipError_t launch_gcm(bool open, const uint8_t* key_dev, int nr, const GcmSegs& segs, int rows,
                      const uint8_t* iv, const uint8_t* aad, int64_t ld_aad, int la, uint8_t* tag,
                      int32_t* ok, uint32_t* partial, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (segs.nseg < 1 || segs.nseg > kGcmMaxSegs || rows > 65535 || la < 0 || la > kGcmMaxAad)
    return hipErrorInvalidValue;
  const int64_t L = segs.end[segs.nseg - 1];
  const int n = (int)((L + 15) / 16);
  const int chain = gcm_chain(rows, n);
  int xpart = 0;
  const int nparts = gcm_parts(n, (la + 15) / 16, chain, &xpart);
  if (nr != 10 && nr != 14) return hipErrorInvalidValue;
  auto kern = open ? (nr == 10 ? k_gcm_blocks<true, 10> : k_gcm_blocks<true, 14>)
                   : (nr == 10 ? k_gcm_blocks<false, 10> : k_gcm_blocks<false, 14>);
  launch_kernel(kern, dim3(nparts, rows), dim3(kGcmStride), 0, s, key_dev, segs, L, n, chain, xpart, iv,
                aad, ld_aad, la, partial, nparts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int fb = (rows + 255) / 256;
  if (open)
    launch_kernel(k_gcm_finish<true>, dim3(fb), dim3(256), 0, s, rows, partial, nparts, tag, ok);
  else
    launch_kernel(k_gcm_finish<false>, dim3(fb), dim3(256), 0, s, rows, partial, nparts, tag, ok);
  return hipGetLastError();
}

}  // namespace sph
