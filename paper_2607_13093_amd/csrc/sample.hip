// Temperature + top-p sampling of each verification row, then the accepted
// draft prefix of each session (eq. 15 with a nucleus cut; Section 5.5).
//
// One 512-thread block per row of fused logits f (fp32, written by the
// endpoint projection, whose per-tile argmax keys also give the row maximum).
// The row is walked in chunks of 256 positions, one per wave iteration (lane
// l holds positions 4l .. 4l+3 of the chunk, loaded as one 16-byte vector),
// so every pass is a short rolled loop of coalesced loads.
//
// Weights.  e = exp((f - fmax) / tau) in fp64 by the table-driven method of
// Tang (ACM TOMS 15(2), 1989): with t = (f - fmax) / (tau ln2) * 64,
// N = rint(t), r = t - N (|r| <= 1/2), e = 2^(N>>6) * 2^((N&63)/64) * 2^(r/64),
// the middle factor from a 64-entry table and 2^(r/64) a degree-5 Taylor
// polynomial (truncation below 4e-17).  Every use of a weight evaluates the
// same operations with contraction off, so it is bit-identical wherever it is
// recomputed.
//
// Exact masses.  Each weight e in [0, 1] becomes E = floor(e * 2^56), held as
// E = a * 2^28 + b (a <= 2^28, b < 2^28).  Masses are exact integer sums of
// E, so the nucleus cut and the inverse CDF are exact for these weights,
// independent of summation order, and the kernel is deterministic.  E misses
// e * 2^56 by less than one unit.
//
//   1. An approximate histogram (fp32 weights, integer atomics) over 4096
//      value buckets of y = (fmax - f)/tau in [0, 40) (the last bucket also
//      takes y >= 40, whose elements each weigh below 5e-18) locates the
//      bucket where the running mass reaches top_p * Z: bucket order is value
//      order, so the nucleus -- the shortest prefix of (p desc, id asc)
//      reaching the target -- ends there.  The window is that bucket, widened
//      by a neighbour where the estimate lies near a bucket edge.
//   2. One exact pass: Z; the masses of the buckets below the window, per
//      segment (runs of consecutive positions, at most 512 per row); the
//      window's elements into an LDS list.  An exact histogram of the list
//      over 128 sub-buckets per bucket finds the sub-bucket holding the cut;
//      one wave ranks its few elements by (key desc, position asc) to find
//      the element completing the nucleus.  The nucleus is
//      {key > T} + {key == T, position <= cut}.
//      Should the window miss the cut or overflow the list, an exact
//      histogram over groups of 4 buckets picks the group and the pass is
//      redone on it; a sub-bucket holding more than 64 elements is ranked by
//      a bitonic sort of the list, and a group with more than 1024 elements
//      goes through an exact radix select over its keys (8 bits per pass),
//      the cut among elements tied at the threshold key being the c-th in id
//      order.
//   3. u = top 24 bits of word 0 of Philox4x32-10 (key = seed halves,
//      counter = (row in session, session, 0, 0)).  The token is the first
//      nucleus member in id order whose running mass M has
//      M * 2^24 > u24 * mass(nucleus): a scan over segment masses picks the
//      segment, one wave scans inside it.
#include "sph_internal.h"

namespace sph {

constexpr int kSThreads = 512;
constexpr int kSWaves = kSThreads / 64;
constexpr int kBuckets = 4096;     // value buckets of (fmax - f)/tau over [0, kYSpan)
constexpr int kBPT = kBuckets / kSThreads;
constexpr int kCoarse = 1024;      // exact fallback histogram: 4 value buckets each
constexpr int kSub = 128;          // sub-buckets per bucket of the window
constexpr int kMaxSub = 4 * kSub;  // window of at most 4 buckets
constexpr int kMaxSeg = kSThreads; // segments per row, one per thread in scans
constexpr int kMaxCand = 1024;     // window elements held in LDS
constexpr int kChunk = 256;        // positions per wave iteration
constexpr int kSegChunks = 4;      // chunks per segment at least
constexpr float kYSpan = 40.0f;
static_assert(kMaxCand == 2 * kSThreads, "two list entries per thread");
static_assert(kCoarse == 2 * kSThreads, "two coarse buckets per thread");
static_assert(kMaxSub == kSThreads, "one sub-bucket per thread");

// 2^(r/64) = exp(r * ln2/64): Taylor coefficients (ln2/64)^k / k!
constexpr double kLn2 = 0.6931471805599453;
constexpr double kL64 = kLn2 / 64.0;
constexpr double kC1 = kL64;
constexpr double kC2 = kL64 * kL64 / 2.0;
constexpr double kC3 = kL64 * kL64 * kL64 / 6.0;
constexpr double kC4 = kL64 * kL64 * kL64 * kL64 / 24.0;
constexpr double kC5 = kL64 * kL64 * kL64 * kL64 * kL64 / 120.0;

// ---------------------------------------------------------------------------
// 128-bit unsigned integers (masses in units of 2^-56)

struct U128 {
  uint64_t lo, hi;
};

__device__ __forceinline__ U128 u128_add(U128 a, U128 b) {
  U128 r;
  r.lo = a.lo + b.lo;
  r.hi = a.hi + b.hi + (r.lo < a.lo ? 1ull : 0ull);
  return r;
}

__device__ __forceinline__ U128 u128_sub(U128 a, U128 b) {
  U128 r;
  r.lo = a.lo - b.lo;
  r.hi = a.hi - b.hi - (a.lo < b.lo ? 1ull : 0ull);
  return r;
}

__device__ __forceinline__ bool u128_lt(U128 a, U128 b) {
  return a.hi < b.hi || (a.hi == b.hi && a.lo < b.lo);
}

__device__ __forceinline__ U128 u128_shl24(U128 a) {
  return U128{a.lo << 24, (a.hi << 24) | (a.lo >> 40)};
}

__device__ __forceinline__ U128 u128_mul32(U128 a, uint32_t m) {
  return U128{a.lo * m, a.hi * m + __umul64hi(a.lo, (uint64_t)m)};
}

// A * 2^28 + B
__device__ __forceinline__ U128 u128_join(uint64_t A, uint64_t B) {
  return u128_add(U128{A << 28, A >> 36}, U128{B, 0ull});
}

__device__ __forceinline__ double u128_to_f64(U128 a) {
  return (double)a.hi * 0x1.0p64 + (double)a.lo;
}

// ceil(x) for finite x >= 0 (x < 2^127)
__device__ U128 u128_ceil(double x) {
  if (!(x > 0.0)) return U128{0ull, 0ull};
  if (x < 1.0) return U128{1ull, 0ull};
  const uint64_t bits = (uint64_t)__double_as_longlong(x);
  const int e = (int)(bits >> 52) - 1023;
  const uint64_t m = (bits & 0xFFFFFFFFFFFFFull) | 0x10000000000000ull;  // x = m * 2^(e-52)
  if (e <= 52) {
    const int sh = 52 - e;
    uint64_t q = m >> sh;
    if ((q << sh) != m) ++q;
    return U128{q, 0ull};
  }
  const int sh = e - 52;
  if (sh < 64) return U128{m << sh, m >> (64 - sh)};
  return U128{0ull, m << (sh - 64)};
}

// E = floor(w * 2^56) = a * 2^28 + b from w28 = w * 2^28 in [0, 2^28].
struct Fix {
  uint32_t a, b;
};

__device__ __forceinline__ Fix fix_of(double w28) {
#pragma clang fp contract(off)
  const uint32_t a = (uint32_t)w28;
  const double r = w28 - (double)a;  // exact, in [0, 1)
  return Fix{a, (uint32_t)(r * 268435456.0)};
}

// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t orderable(float v) {
  v = v + 0.0f;  // -0 -> +0
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_orderable(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}

// exp((x - fmax) / tau) * 2^28 with kk = 64 / (tau ln2), c0 = -fmax * kk.
__device__ __forceinline__ double weight28(float x, double kk, double c0,
                                           const double* __restrict__ tab) {
#pragma clang fp contract(off)
  double t = fma((double)x, kk, c0);
  t = fmin(fmax(t, -90000.0), 0.0);  // 2^(-90000/64) is zero in fp64; x <= fmax
  const double nn = rint(t);
  const double r = t - nn;  // exact, |r| <= 1/2
  const double p = fma(r, fma(r, fma(r, fma(r, fma(r, kC5, kC4), kC3), kC2), kC1), 1.0);
  const int j = (int)nn;
  return ldexp(tab[j & 63] * p, (j >> 6) + 28);
}

// (fmax - x) * kb with kb = kBuckets / (kYSpan tau): bucket units, >= 0.
__device__ __forceinline__ float ypos(float x, float vmax, float kb) {
#pragma clang fp contract(off)
  return (vmax - x) * kb;
}

// Value bucket: floor(ypos), the last bucket taking everything beyond.
// Non-decreasing as x decreases.
__device__ __forceinline__ int bucket_of(float y) {
  return (int)fminf(y, (float)(kBuckets - 1));
}

// Sub-bucket: floor(ypos * kSub) (exact scaling), consistent with bucket_of:
// bucket b holds sub-buckets [kSub b, kSub b + kSub - 1].
__device__ __forceinline__ int subbucket_of(float y) {
  return (int)fminf(y * (float)kSub, (float)(kSub * kBuckets - 1));
}

// Philox4x32-10 (Salmon et al., SC'11), word 0 of the output block.
__device__ uint32_t philox_x0(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                              uint32_t k1) {
  constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += W0;
      k1 += W1;
    }
    const uint32_t hi0 = __umulhi(M0, c0), lo0 = M0 * c0;
    const uint32_t hi1 = __umulhi(M1, c2), lo1 = M1 * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return c0;
}

// ---------------------------------------------------------------------------
// wave and block primitives (fixed order)

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t x, int o) {
  const uint32_t lo = __shfl_up((uint32_t)x, o, 64);
  const uint32_t hi = __shfl_up((uint32_t)(x >> 32), o, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t x, int src) {
  const uint32_t lo = __shfl((uint32_t)x, src, 64);
  const uint32_t hi = __shfl((uint32_t)(x >> 32), src, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int o) {
  const uint32_t lo = __shfl_xor((uint32_t)x, o, 64);
  const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), o, 64);
  return ((uint64_t)hi << 32) | lo;
}

// Sum over the wave, in every lane, without the LDS crossbar: the 32- and
// 16-lane steps swap register halves with v_permlane32_swap /
// v_permlane16_swap (both results summed), then DPP rotations by 8, 4, 2
// and 1 lanes inside each 16-lane row finish the sum.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  return ((uint64_t)dpp_u32<CTRL>((uint32_t)(v >> 32)) << 32) | dpp_u32<CTRL>((uint32_t)v);
}
template <bool W32>
__device__ __forceinline__ uint64_t swap_sum_u64(uint64_t v) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  const auto l = W32 ? __builtin_amdgcn_permlane32_swap(lo, lo, false, false)
                     : __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
  const auto h = W32 ? __builtin_amdgcn_permlane32_swap(hi, hi, false, false)
                     : __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
  return (((uint64_t)h[0] << 32) | l[0]) + (((uint64_t)h[1] << 32) | l[1]);
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  v = swap_sum_u64<true>(v);
  v = swap_sum_u64<false>(v);
  v += dpp_u64<0x128>(v);  // row_ror:8
  v += dpp_u64<0x124>(v);  // row_ror:4
  v += dpp_u64<0x122>(v);  // row_ror:2
  v += dpp_u64<0x121>(v);  // row_ror:1
  return v;
}

__device__ __forceinline__ U128 wave_inscan_u128(U128 v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const U128 y{shfl_up_u64(v.lo, o), shfl_up_u64(v.hi, o)};
    if (lane >= o) v = u128_add(v, y);
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_inscan_u32(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(v, o, 64);
    if (lane >= o) v += y;
  }
  return v;
}

struct SampleShared {
  union {
    unsigned long long hf[kBuckets + 64];  // approximate bucket masses (units of 2^-32)
    struct {
      uint64_t key[kMaxCand];  // (~orderable key) << 32 | position: ascending = nucleus order
      uint64_t a[kMaxCand];
      uint64_t b[kMaxCand];
      uint64_t sa[kMaxSub];  // exact sub-bucket masses of the window
      uint64_t sb[kMaxSub];
      uint32_t scnt[kMaxSub];
    } c;
    struct {
      uint64_t a[kCoarse + 64];  // exact group masses, 64 per-lane spill slots
      uint64_t b[kCoarse + 64];
      uint32_t cnt[256];  // element counts of the key passes
    } h;
  } u;
  uint64_t seg_a[kMaxSeg];  // nucleus mass per segment
  uint64_t seg_b[kMaxSeg];
  uint32_t seg_t[kMaxSeg];  // elements tied at the threshold key per segment
  uint64_t wkey[64];        // the crossing sub-bucket's elements
  uint64_t wa[64];
  uint64_t wb[64];
  double tab[64];
  U128 xred[kSWaves];
  double dred[kSWaves];
  uint64_t kred[kSWaves];
  uint32_t ured[kSWaves];
  U128 above, claim_base;
  uint32_t tie_base, T;
  int32_t bsel, lo, hi, ncand, cut_idx, cut_pos, claim_seg, tie_seg;
};

__device__ unsigned long long block_max_u64(unsigned long long v, SampleShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = max(v, (unsigned long long)shfl_xor_u64(v, o));
  __syncthreads();
  if (lane == 0) sh.kred[wave] = v;
  __syncthreads();
  unsigned long long r = sh.kred[0];
  for (int w = 1; w < kSWaves; ++w) r = max(r, (unsigned long long)sh.kred[w]);
  return r;
}

// Exclusive prefix sums over threads (thread order); *total = sum.
__device__ U128 block_exscan_u128(U128 v, SampleShared& sh, U128* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const U128 inc = wave_inscan_u128(v);
  __syncthreads();
  if (lane == 63) sh.xred[wave] = inc;
  __syncthreads();
  U128 base{0ull, 0ull}, tot{0ull, 0ull};
  for (int w = 0; w < kSWaves; ++w) {
    if (w < wave) base = u128_add(base, sh.xred[w]);
    tot = u128_add(tot, sh.xred[w]);
  }
  *total = tot;
  return u128_add(base, u128_sub(inc, v));
}

__device__ double block_exscan_f64(double v, SampleShared& sh, double* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y =
        __longlong_as_double((long long)shfl_up_u64((uint64_t)__double_as_longlong(inc), o));
    if (lane >= o) inc += y;
  }
  __syncthreads();
  if (lane == 63) sh.dred[wave] = inc;
  __syncthreads();
  double base = 0.0, tot = 0.0;
  for (int w = 0; w < kSWaves; ++w) {
    if (w < wave) base += sh.dred[w];
    tot += sh.dred[w];
  }
  *total = tot;
  return base + inc - v;
}

__device__ uint32_t block_exscan_u32(uint32_t v, SampleShared& sh, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t inc = wave_inscan_u32(v);
  __syncthreads();
  if (lane == 63) sh.ured[wave] = inc;
  __syncthreads();
  uint32_t base = 0, tot = 0;
  for (int w = 0; w < kSWaves; ++w) {
    if (w < wave) base += sh.ured[w];
    tot += sh.ured[w];
  }
  *total = tot;
  return base + inc - v;
}

__device__ __forceinline__ U128 block_sum_u128(U128 v, SampleShared& sh) {
  U128 tot;
  block_exscan_u128(v, sh, &tot);
  return tot;
}

// The lane's four positions p .. p+3 of a chunk; positions past the row are
// invalid and not read.
template <bool VEC>
__device__ __forceinline__ void load4(const float* __restrict__ row, int n, int p, float (&x)[4],
                                      bool (&v)[4]) {
  if (VEC && p + 3 < n) {
    const float4 q = *reinterpret_cast<const float4*>(row + p);
    x[0] = q.x;
    x[1] = q.y;
    x[2] = q.z;
    x[3] = q.w;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = true;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = p + e < n;
      x[e] = v[e] ? row[p + e] : 0.0f;
    }
  }
}

// fn(q, p, x, v) on every chunk q of the row, chunks dealt to waves in turn,
// two chunks loaded ahead per wave iteration.
template <bool VEC, class F>
__device__ __forceinline__ void for_chunks(const float* __restrict__ row, int n, int NC, F&& fn) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int q = wave; q < NC; q += 2 * kSWaves) {
    const int q2 = q + kSWaves;
    float x0[4], x1[4];
    bool v0[4], v1[4];
    load4<VEC>(row, n, q * kChunk + 4 * lane, x0, v0);
    load4<VEC>(row, n, q2 * kChunk + 4 * lane, x1, v1);
    fn(q, q * kChunk + 4 * lane, x0, v0);
    if (q2 < NC) fn(q2, q2 * kChunk + 4 * lane, x1, v1);
  }
}

// fn(q, p, x, v) on every chunk q of the row, each wave on one contiguous
// range of chunks (so that a segment's chunks mostly fall to one wave), two
// chunks loaded per iteration.
template <bool VEC, class F>
__device__ __forceinline__ void for_chunks_contig(const float* __restrict__ row, int n, int NC, F&& fn) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int per = (NC + kSWaves - 1) / kSWaves;
  const int q1 = min(NC, (wave + 1) * per);
  for (int q = wave * per; q < q1; q += 2) {
    float x0[4], x1[4];
    bool v0[4], v1[4];
    load4<VEC>(row, n, q * kChunk + 4 * lane, x0, v0);
    if (q + 1 < q1) load4<VEC>(row, n, (q + 1) * kChunk + 4 * lane, x1, v1);
    fn(q, q * kChunk + 4 * lane, x0, v0);
    if (q + 1 < q1) fn(q + 1, (q + 1) * kChunk + 4 * lane, x1, v1);
  }
}

// VEC: rows start 16-byte aligned (n % 4 == 0), positions load as float4.
template <bool VEC>
__global__ __launch_bounds__(kSThreads) __attribute__((amdgpu_waves_per_eu(6))) void k_sample(
    const float* __restrict__ f, int n, const unsigned long long* __restrict__ best, int nblk,
    const int32_t* __restrict__ ids, int R, float temperature, float top_p, uint32_t seed_lo,
    uint32_t seed_hi, int32_t* __restrict__ tokens) {
  __shared__ SampleShared sh;
  const int m = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* row = f + (int64_t)m * n;
  // segments of G positions (a multiple of the chunk, at least kSegChunks
  // chunks), at most kMaxSeg of them
  const int G = kChunk * max(kSegChunks, (n + kChunk * kMaxSeg - 1) / (kChunk * kMaxSeg));
  const int NS = (n + G - 1) / G;
  const int NC = (n + kChunk - 1) / kChunk;

  if (t < 64) sh.tab[t] = exp2((double)t * (1.0 / 64.0));
  sh.seg_a[t] = 0ull;
  sh.seg_b[t] = 0ull;
  sh.seg_t[t] = 0u;
  if (t == 0) {
    sh.bsel = -1;
    sh.ncand = 0;
    sh.cut_idx = -1;
    sh.cut_pos = n;
    sh.claim_seg = -1;
    sh.tie_seg = -1;
    sh.T = 0u;
  }
  // row maximum from the projection's per-tile argmax keys
  unsigned long long kmax = 0ull;
  for (int i = t; i < nblk; i += kSThreads) kmax = max(kmax, best[(int64_t)m * kMaxBlocks + i]);
  kmax = block_max_u64(kmax, sh);  // its barriers also publish the table and the zeroed state
  const float vmax = from_orderable((uint32_t)(kmax >> 32));
  const double kk = 64.0 / (kLn2 * (double)temperature);
  const double c0 = -(double)vmax * kk;
  const float kb = (float)kBuckets / (kYSpan * temperature);
  const double* tab = sh.tab;
  auto fix = [&](float x) { return fix_of(weight28(x, kk, c0, tab)); };
  auto member = [&](float x, int pos, uint32_t T, int cut) {
    const uint32_t k = orderable(x);
    return k > T || (k == T && pos <= cut);
  };

  // Exact pass with the window [lo, hi]: segment masses of the buckets below
  // lo, the window's elements into the list.  Returns the total mass Z.  A
  // wave's chunks are contiguous, so each lane sums its share of a segment
  // and the wave reduces it once per segment (one wave-wide sum per chunk
  // cost a quarter of the pass); one vote per chunk skips the list code
  // where no element of the chunk falls in the window.
  auto collect = [&](int lo, int hi) -> U128 {
    uint64_t za = 0ull, zb = 0ull;
    uint64_t sa = 0ull, sbm = 0ull;  // the lane's masses below the window in segment cur
    int cur = -1;
    auto flush = [&]() {
      const uint64_t A = wave_sum_u64(sa), B = wave_sum_u64(sbm);
      if (lane == 0 && (A | B)) {
        atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_a[cur]), (unsigned long long)A);
        atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_b[cur]), (unsigned long long)B);
      }
      sa = 0ull;
      sbm = 0ull;
    };
    for_chunks_contig<VEC>(row, n, NC, [&](int q, int p, const float (&x)[4], const bool (&v)[4]) {
      const int sg = q * kChunk / G;
      if (sg != cur) {
        if (cur >= 0) flush();
        cur = sg;
      }
      uint32_t ca = 0u, cb = 0u, ma = 0u, mb = 0u;  // four weights of at most 2^28 each
      Fix w[4];
      bool cand[4];
      bool anyc = false;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w[e] = fix(x[e]);
        const int b = bucket_of(ypos(x[e], vmax, kb));
        ca += v[e] ? w[e].a : 0u;
        cb += v[e] ? w[e].b : 0u;
        const bool mem = v[e] && b < lo;
        ma += mem ? w[e].a : 0u;
        mb += mem ? w[e].b : 0u;
        cand[e] = v[e] && b >= lo && b <= hi;
        anyc |= cand[e];
      }
      if (__ballot(anyc)) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint64_t bal = __ballot(cand[e]);
          if (bal) {
            const int leader = __ffsll((unsigned long long)bal) - 1;
            int base = 0;
            if (lane == leader) base = atomicAdd(&sh.ncand, __popcll(bal));
            base = __shfl(base, leader, 64);
            if (cand[e]) {
              const int slot = base + __popcll(bal & ((1ull << lane) - 1ull));
              if (slot < kMaxCand) {
                const Fix wr = w[e];
                sh.u.c.key[slot] = ((uint64_t)(~orderable(x[e])) << 32) | (uint32_t)(p + e);
                sh.u.c.a[slot] = wr.a;
                sh.u.c.b[slot] = wr.b;
              }
            }
          }
        }
      }
      za += ca;
      zb += cb;
      sa += ma;
      sbm += mb;
    });
    if (cur >= 0) flush();
    return block_sum_u128(u128_join(za, zb), sh);  // barriers: segments and list complete
  };
  const bool all = !(top_p < 1.0f);
  int lo = kBuckets, hi = kBuckets - 1;  // all: every bucket below lo, no window
  if (!all) {
    // 1. approximate histogram (fp32 weights in units of 2^-32) -> window
    for (int b = t; b < kBuckets + 64; b += kSThreads) sh.u.hf[b] = 0ull;
    __syncthreads();
    const float c32 = 1.4426950408889634f / temperature;
    for_chunks<VEC>(row, n, NC, [&](int, int, const float (&x)[4], const bool (&v)[4]) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float y = ypos(x[e], vmax, kb);
        const float w = exp2f((x[e] - vmax) * c32);
        int b = bucket_of(y);
        if (!v[e] || b == kBuckets - 1) b = kBuckets + lane;
        atomicAdd(&sh.u.hf[b], v[e] ? (unsigned long long)(uint32_t)(w * 4294967040.0f) : 0ull);
      }
    });
    __syncthreads();
    if (wave == 0) {
      const uint64_t tail = wave_sum_u64(sh.u.hf[kBuckets + lane]);
      if (lane == 0) sh.u.hf[kBuckets - 1] += tail;
    }
    __syncthreads();
    double d[kBPT];
    double dl = 0.0;
#pragma unroll
    for (int i = 0; i < kBPT; ++i) {
      d[i] = (double)sh.u.hf[kBPT * t + i];
      dl += d[i];
    }
    double ztot;
    double acc = block_exscan_f64(dl, sh, &ztot);
    const double need_a = (double)top_p * ztot;
    // error of the estimate: fp32 exponent and exp2 rounding, truncation
    const double slack = 1e-5 * ztot + 2.0 * (double)n;
#pragma unroll
    for (int i = 0; i < kBPT; ++i) {
      if (acc < need_a && acc + d[i] >= need_a) {
        const int b = kBPT * t + i;
        sh.lo = (acc >= need_a - slack && b > 0) ? b - 1 : b;
        sh.hi = (acc + d[i] <= need_a + slack && b < kBuckets - 1) ? b + 1 : b;
        sh.bsel = b;
      }
      acc += d[i];
    }
    __syncthreads();
    if (sh.bsel >= 0) {
      lo = sh.lo;
      hi = sh.hi;
    } else {
      lo = kBuckets - 2;
      hi = kBuckets - 1;
    }
    __syncthreads();
  }

  // 2. exact pass: Z, segment masses below the window, the window's list
  const U128 Z = collect(lo, hi);
  if (!all) {
    U128 need = u128_ceil((double)top_p * u128_to_f64(Z));
    if (need.lo == 0ull && need.hi == 0ull) need.lo = 1ull;
    U128 above = block_sum_u128(u128_join(sh.seg_a[t], sh.seg_b[t]), sh);
    int nc = sh.ncand;
    U128 wmass{0ull, 0ull};
    if (nc <= kMaxCand) {
      U128 cl{0ull, 0ull};
      for (int i = t; i < nc; i += kSThreads) cl = u128_add(cl, u128_join(sh.u.c.a[i], sh.u.c.b[i]));
      wmass = block_sum_u128(cl, sh);
    }
    if (nc > kMaxCand || !u128_lt(above, need) || u128_lt(u128_add(above, wmass), need)) {
      // the window missed the cut or overflowed the list: exact histogram
      // over groups of 4 buckets, then the exact pass over that group
      __syncthreads();
      for (int b = t; b < kCoarse + 64; b += kSThreads) {
        sh.u.h.a[b] = 0ull;
        sh.u.h.b[b] = 0ull;
      }
      if (t == 0) {
        sh.bsel = -1;
        sh.ncand = 0;
      }
      sh.seg_a[t] = 0ull;
      sh.seg_b[t] = 0ull;
      __syncthreads();
      for_chunks<VEC>(row, n, NC, [&](int, int, const float (&x)[4], const bool (&v)[4]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const Fix w = fix(x[e]);
          int b = bucket_of(ypos(x[e], vmax, kb)) >> 2;
          if (!v[e] || b == kCoarse - 1) b = kCoarse + lane;
          atomicAdd(reinterpret_cast<unsigned long long*>(&sh.u.h.a[b]),
                    (unsigned long long)(v[e] ? w.a : 0u));
          atomicAdd(reinterpret_cast<unsigned long long*>(&sh.u.h.b[b]),
                    (unsigned long long)(v[e] ? w.b : 0u));
        }
      });
      __syncthreads();
      if (wave == 0) {
        const uint64_t ta = wave_sum_u64(sh.u.h.a[kCoarse + lane]);
        const uint64_t tb = wave_sum_u64(sh.u.h.b[kCoarse + lane]);
        if (lane == 0) {
          sh.u.h.a[kCoarse - 1] += ta;
          sh.u.h.b[kCoarse - 1] += tb;
        }
      }
      __syncthreads();
      const U128 s0 = u128_join(sh.u.h.a[2 * t], sh.u.h.b[2 * t]);
      const U128 s1 = u128_join(sh.u.h.a[2 * t + 1], sh.u.h.b[2 * t + 1]);
      U128 tot;
      const U128 x0 = block_exscan_u128(u128_add(s0, s1), sh, &tot);
      const U128 x1 = u128_add(x0, s0);
      if (u128_lt(x0, need) && !u128_lt(x1, need)) sh.bsel = 2 * t;
      if (u128_lt(x1, need) && !u128_lt(u128_add(x1, s1), need)) sh.bsel = 2 * t + 1;
      __syncthreads();
      const int cg = max(sh.bsel, 0);
      lo = 4 * cg;
      hi = 4 * cg + 3;
      __syncthreads();
      collect(lo, hi);
      above = block_sum_u128(u128_join(sh.seg_a[t], sh.seg_b[t]), sh);
      nc = sh.ncand;
    }

    if (nc <= kMaxCand) {
      // exact histogram of the list over sub-buckets of the window
      const int nsub = kSub * (hi - lo + 1);
      sh.u.c.sa[t] = 0ull;
      sh.u.c.sb[t] = 0ull;
      sh.u.c.scnt[t] = 0u;
      if (t == 0) sh.bsel = -1;
      __syncthreads();
      auto sub_of = [&](uint64_t key) {
        const float x = from_orderable(~(uint32_t)(key >> 32));
        return min(max(subbucket_of(ypos(x, vmax, kb)) - kSub * lo, 0), nsub - 1);
      };
      for (int i = t; i < nc; i += kSThreads) {
        const int s = sub_of(sh.u.c.key[i]);
        atomicAdd(reinterpret_cast<unsigned long long*>(&sh.u.c.sa[s]),
                  (unsigned long long)sh.u.c.a[i]);
        atomicAdd(reinterpret_cast<unsigned long long*>(&sh.u.c.sb[s]),
                  (unsigned long long)sh.u.c.b[i]);
        atomicAdd(&sh.u.c.scnt[s], 1u);
      }
      __syncthreads();
      const U128 st = u128_join(sh.u.c.sa[t], sh.u.c.sb[t]);
      U128 tot;
      const U128 sx = u128_add(above, block_exscan_u128(st, sh, &tot));
      if (t < nsub && u128_lt(sx, need) && !u128_lt(u128_add(sx, st), need)) {
        sh.bsel = t;
        sh.above = sx;
      }
      __syncthreads();
      const int ss = max(sh.bsel, 0);
      const U128 as = sh.above;
      const uint32_t cs = sh.u.c.scnt[ss];
      if (cs <= 64u) {
        if (wave == 0) {
          // gather sub-bucket ss, then rank it by (key desc, position asc)
          int got = 0;
          for (int base = 0; base < nc; base += 64) {
            const int i = base + lane;
            const bool in = i < nc && sub_of(sh.u.c.key[i]) == ss;
            const uint64_t bal = __ballot(in);
            if (in) {
              const int slot = got + __popcll(bal & ((1ull << lane) - 1ull));
              sh.wkey[slot] = sh.u.c.key[i];
              sh.wa[slot] = sh.u.c.a[i];
              sh.wb[slot] = sh.u.c.b[i];
            }
            got += __popcll(bal);
          }
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          if (lane < got) {
            const uint64_t kj = sh.wkey[lane];
            uint64_t A = 0ull, B = 0ull;
            for (int i = 0; i < got; ++i) {
              const bool before = sh.wkey[i] < kj;
              A += before ? sh.wa[i] : 0ull;
              B += before ? sh.wb[i] : 0ull;
            }
            const U128 ex = u128_add(as, u128_join(A, B));
            const U128 in = u128_add(ex, u128_join(sh.wa[lane], sh.wb[lane]));
            if (u128_lt(ex, need) && !u128_lt(in, need)) {
              sh.T = ~(uint32_t)(kj >> 32);
              sh.cut_pos = (int)(uint32_t)kj;
            }
          }
        }
        __syncthreads();
        // members of the window: sub-buckets before ss, and ss up to the cut
        const uint64_t kc = ((uint64_t)(~sh.T) << 32) | (uint32_t)sh.cut_pos;
        for (int i = t; i < nc; i += kSThreads) {
          const uint64_t key = sh.u.c.key[i];
          const int s = sub_of(key);
          if (s < ss || (s == ss && key <= kc)) {
            const int pos = (int)(uint32_t)key;
            atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_a[pos / G]),
                      (unsigned long long)sh.u.c.a[i]);
            atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_b[pos / G]),
                      (unsigned long long)sh.u.c.b[i]);
          }
        }
      } else {
        // a crowded sub-bucket: bitonic sort of the list, scan, cut
        int P = 1;
        while (P < nc) P <<= 1;
        for (int i = nc + t; i < P; i += kSThreads) {
          sh.u.c.key[i] = ~0ull;
          sh.u.c.a[i] = 0ull;
          sh.u.c.b[i] = 0ull;
        }
        __syncthreads();
        for (int k = 2; k <= P; k <<= 1) {
          for (int j = k >> 1; j > 0; j >>= 1) {
            if (t < P / 2) {
              const int i = 2 * t - (t & (j - 1));
              const int l = i + j;
              const uint64_t ki = sh.u.c.key[i], kl = sh.u.c.key[l];
              if ((ki > kl) == ((i & k) == 0)) {
                sh.u.c.key[i] = kl;
                sh.u.c.key[l] = ki;
                const uint64_t ai = sh.u.c.a[i], bi = sh.u.c.b[i];
                sh.u.c.a[i] = sh.u.c.a[l];
                sh.u.c.b[i] = sh.u.c.b[l];
                sh.u.c.a[l] = ai;
                sh.u.c.b[l] = bi;
              }
            }
            __syncthreads();
          }
        }
        const int i0 = 2 * t, i1 = 2 * t + 1;
        const U128 e0 = i0 < nc ? u128_join(sh.u.c.a[i0], sh.u.c.b[i0]) : U128{0ull, 0ull};
        const U128 e1 = i1 < nc ? u128_join(sh.u.c.a[i1], sh.u.c.b[i1]) : U128{0ull, 0ull};
        U128 tot2;
        const U128 ex0 = u128_add(above, block_exscan_u128(u128_add(e0, e1), sh, &tot2));
        const U128 ex1 = u128_add(ex0, e0);
        if (i0 < nc && u128_lt(ex0, need) && !u128_lt(ex1, need)) sh.cut_idx = i0;
        if (i1 < nc && u128_lt(ex1, need) && !u128_lt(u128_add(ex1, e1), need)) sh.cut_idx = i1;
        __syncthreads();
        const int jc = sh.cut_idx;
        for (int i = t; i <= jc; i += kSThreads) {
          const int pos = (int)(uint32_t)sh.u.c.key[i];
          atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_a[pos / G]),
                    (unsigned long long)sh.u.c.a[i]);
          atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_b[pos / G]),
                    (unsigned long long)sh.u.c.b[i]);
        }
        if (t == 0 && jc >= 0) {
          sh.T = ~(uint32_t)(sh.u.c.key[jc] >> 32);
          sh.cut_pos = (int)(uint32_t)sh.u.c.key[jc];
        }
      }
    } else {
      // exact radix select, 8 bits per pass, on the keys of the window
      auto in_window = [&](float x) {
        const int b = bucket_of(ypos(x, vmax, kb));
        return b >= lo && b <= hi;
      };
      uint32_t Tk = 0u, kmask = 0u, nt = 0u;
      U128 ab = above;
      for (int shift = 24; shift >= 0; shift -= 8) {
        __syncthreads();  // earlier readers of the histogram are done
        if (t < 256) {
          sh.u.h.a[t] = 0ull;
          sh.u.h.b[t] = 0ull;
          sh.u.h.cnt[t] = 0u;
        }
        if (t == 0) sh.bsel = -1;
        __syncthreads();
        for_chunks<VEC>(row, n, NC, [&](int, int, const float (&x)[4], const bool (&v)[4]) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t key = orderable(x[e]);
            if (v[e] && in_window(x[e]) && (key & kmask) == Tk) {
              const int b = (int)((key >> shift) & 255u);
              const Fix w = fix(x[e]);
              atomicAdd(reinterpret_cast<unsigned long long*>(&sh.u.h.a[b]),
                        (unsigned long long)w.a);
              atomicAdd(reinterpret_cast<unsigned long long*>(&sh.u.h.b[b]),
                        (unsigned long long)w.b);
              atomicAdd(&sh.u.h.cnt[b], 1u);
            }
          }
        });
        __syncthreads();
        // thread t < 256 owns key bucket 255 - t: descending keys
        const U128 ks =
            t < 256 ? u128_join(sh.u.h.a[255 - t], sh.u.h.b[255 - t]) : U128{0ull, 0ull};
        U128 ktot;
        const U128 kacc = u128_add(ab, block_exscan_u128(ks, sh, &ktot));
        if (t < 256 && u128_lt(kacc, need) && !u128_lt(u128_add(kacc, ks), need)) {
          sh.bsel = 255 - t;
          sh.above = kacc;
        }
        __syncthreads();
        const int sel = max(sh.bsel, 0);
        ab = sh.bsel >= 0 ? sh.above : ab;
        nt = sh.u.h.cnt[sel];
        Tk |= (uint32_t)sel << shift;
        kmask |= 255u << shift;
      }
      // the c-th element tied at Tk in id order completes the nucleus:
      // smallest c >= 1 with ab + c * E(Tk) >= need
      const Fix wt = fix(from_orderable(Tk));
      const U128 WT = u128_join(wt.a, wt.b);
      const double cd = ceil(u128_to_f64(u128_sub(need, ab)) / u128_to_f64(WT));
      uint32_t c = cd < 1.0 ? 1u : (cd > (double)nt ? nt : (uint32_t)cd);
      while (c > 1u && !u128_lt(u128_add(ab, u128_mul32(WT, c - 1u)), need)) --c;
      while (c < nt && u128_lt(u128_add(ab, u128_mul32(WT, c)), need)) ++c;
      // ties per segment, then the segment and the lane holding the c-th
      for_chunks<VEC>(row, n, NC, [&](int q, int, const float (&x)[4], const bool (&v)[4]) {
        uint32_t ties = 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e) ties += (v[e] && orderable(x[e]) == Tk) ? 1u : 0u;
        ties = (uint32_t)wave_sum_u64(ties);
        if (lane == 0 && ties) atomicAdd(&sh.seg_t[q * kChunk / G], ties);
      });
      __syncthreads();
      const uint32_t tc = t < NS ? sh.seg_t[t] : 0u;
      uint32_t ttot;
      const uint32_t tb = block_exscan_u32(tc, sh, &ttot);
      if (tb < c && c <= tb + tc) {
        sh.tie_seg = t;
        sh.tie_base = tb;
      }
      __syncthreads();
      if (wave == 0 && sh.tie_seg >= 0) {
        const int sg = sh.tie_seg;
        uint32_t run = sh.tie_base;
        const int end = min(n, (sg + 1) * G);
        for (int cb = sg * G; cb < end; cb += kChunk) {
          const int p = cb + 4 * lane;
          float x[4];
          bool v[4];
          load4<VEC>(row, n, p, x, v);
          bool tie[4];
          uint32_t lt = 0u;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            tie[e] = v[e] && orderable(x[e]) == Tk;
            lt += tie[e] ? 1u : 0u;
          }
          const uint32_t inc = wave_inscan_u32(lt);
          uint32_t seen = run + inc - lt;
          int hit = -1;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (tie[e] && ++seen == c && hit < 0) hit = p + e;
          const uint64_t bal = __ballot(hit >= 0);
          if (bal) {
            const int pos = __shfl(hit, __ffsll((unsigned long long)bal) - 1, 64);
            if (lane == 0) {
              sh.T = Tk;
              sh.cut_pos = pos;
            }
            break;
          }
          run += __shfl(inc, 63, 64);
        }
      }
      __syncthreads();
      // members of the window
      const uint32_t Tw = sh.T;
      const int cw = sh.cut_pos;
      for_chunks<VEC>(row, n, NC, [&](int q, int p, const float (&x)[4], const bool (&v)[4]) {
        uint64_t A = 0ull, B = 0ull;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (v[e] && in_window(x[e]) && member(x[e], p + e, Tw, cw)) {
            const Fix w = fix(x[e]);
            A += w.a;
            B += w.b;
          }
        }
        A = wave_sum_u64(A);
        B = wave_sum_u64(B);
        if (lane == 0 && (A | B)) {
          const int sg = q * kChunk / G;
          atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_a[sg]), (unsigned long long)A);
          atomicAdd(reinterpret_cast<unsigned long long*>(&sh.seg_b[sg]), (unsigned long long)B);
        }
      });
    }
    __syncthreads();
  }
  // Nucleus: key > T, or key == T and position <= cut (T = 0, cut = n: all).
  const uint32_t T = sh.T;
  const int cut = sh.cut_pos;

  // 3. segment masses in id order, then the inverse CDF inside one segment
  const U128 sm = t < NS ? u128_join(sh.seg_a[t], sh.seg_b[t]) : U128{0ull, 0ull};
  U128 mass;
  const U128 sb = block_exscan_u128(sm, sh, &mass);
  const uint32_t s_idx = (uint32_t)(m / R), r_idx = (uint32_t)(m % R);
  const uint32_t u24 = philox_x0(r_idx, s_idx, 0u, 0u, seed_lo, seed_hi) >> 8;
  const U128 target = u128_mul32(mass, u24);
  if (!u128_lt(target, u128_shl24(sb)) && u128_lt(target, u128_shl24(u128_add(sb, sm)))) {
    sh.claim_seg = t;
    sh.claim_base = sb;
  }
  __syncthreads();
  if (wave == 0) {
    const int sg = sh.claim_seg;
    int pick = -1;
    if (sg >= 0) {
      U128 run = sh.claim_base;
      const int end = min(n, (sg + 1) * G);
      // the segment's chunks in groups of kSegChunks, a group's loads issued
      // together
      for (int cg = sg * G; cg < end && pick < 0; cg += kSegChunks * kChunk) {
      float xg[kSegChunks][4];
      bool vg[kSegChunks][4];
#pragma unroll
      for (int c = 0; c < kSegChunks; ++c) load4<VEC>(row, n, cg + c * kChunk + 4 * lane, xg[c], vg[c]);
#pragma unroll
      for (int c = 0; c < kSegChunks; ++c) {
        const int cb = cg + c * kChunk;
        if (cb >= end || pick >= 0) break;
        const int p = cb + 4 * lane;
        float x[4];
        bool v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[e] = xg[c][e];
          v[e] = vg[c][e];
        }
        U128 li[4];
        U128 l{0ull, 0ull};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (v[e] && member(x[e], p + e, T, cut)) {
            const Fix w = fix(x[e]);
            l = u128_add(l, u128_join(w.a, w.b));
          }
          li[e] = l;
        }
        const U128 inc = wave_inscan_u128(l);
        const U128 lb = u128_add(run, u128_sub(inc, l));
        int hit = -1;
#pragma unroll
        for (int e = 3; e >= 0; --e)
          if (u128_lt(target, u128_shl24(u128_add(lb, li[e])))) hit = e;
        const uint64_t bal = __ballot(hit >= 0);
        if (bal) {
          const int src = __ffsll((unsigned long long)bal) - 1;
          pick = cb + 4 * src + __shfl(hit, src, 64);
        }
        run = u128_add(run, U128{shfl_u64(inc.lo, 63), shfl_u64(inc.hi, 63)});
      }
      }
    }
    if (lane == 0) tokens[m] = ids[pick >= 0 ? pick : 0];
  }
}

__global__ void k_accept(const int32_t* __restrict__ tokens, const int32_t* __restrict__ drafts,
                         int n_sessions, int R, int32_t* __restrict__ accept) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_sessions) return;
  const int kd = R - 1;
  int a = 0;
  bool run = true;
  // tokens and drafts are loaded eight at a time, before any comparison
  for (int b = 0; b < kd && run; b += 8) {
    int32_t t[8], d[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const bool ok = b + u < kd;
      t[u] = ok ? tokens[(int64_t)s * R + b + u] : 0;
      d[u] = ok ? drafts[(int64_t)s * kd + b + u] : 0;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (run && b + u < kd && t[u] == d[u]) ++a;
      else run = false;
    }
  }
  accept[s] = a;
}

hipError_t launch_sample(const float* f, int M, int n, const unsigned long long* best, int nblk,
                         const int32_t* ids, int R, float temperature, float top_p, uint64_t seed,
                         int32_t* tokens, hipStream_t s) {
  if (n < 1 || nblk < 1 || nblk > kMaxBlocks) return hipErrorInvalidValue;
  if ((int64_t)(n + kChunk * kMaxSeg - 1) / (kChunk * kMaxSeg) * kChunk * kMaxSeg >= (1ll << 31))
    return hipErrorInvalidValue;
  const uint32_t lo = (uint32_t)seed, hi = (uint32_t)(seed >> 32);
  const bool vec = n % 4 == 0 && (reinterpret_cast<uintptr_t>(f) & 15u) == 0;
  if (vec)
    launch_kernel(k_sample<true>, dim3(M), dim3(kSThreads), 0, s, f, n, best, nblk, ids, R,
                       temperature, top_p, lo, hi, tokens);
  else
    launch_kernel(k_sample<false>, dim3(M), dim3(kSThreads), 0, s, f, n, best, nblk, ids, R,
                       temperature, top_p, lo, hi, tokens);
  return hipGetLastError();
}

hipError_t launch_accept(const int32_t* tokens, const int32_t* drafts, int n_sessions, int R,
                         int32_t* accept, hipStream_t s) {
  launch_kernel(k_accept, dim3((n_sessions + 255) / 256), dim3(256), 0, s, tokens, drafts,
                     n_sessions, R, accept);
  return hipGetLastError();
}

}  // namespace sph
