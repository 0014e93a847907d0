// Temperature + top-p sampling of each verification row, then the accepted
// draft prefix of each session (eq. 15 with a nucleus cut; Section 5.5).
//
// One 1024-thread block per row of fused logits f (fp32, written by the
// endpoint projection).  Thread t holds the contiguous positions
// [t*CH, (t+1)*CH) of the row, i.e. a run of ascending vocabulary ids, so
// every id-order quantity is a per-thread sequential pass plus a block scan.
//
//   1. fmax = max f; softmax weights e_j = exp((f_j - fmax) / tau) in fp64,
//      Z = sum e (per-thread sequential sums, fixed-order tree).
//   2. Nucleus = shortest prefix of (p desc, id asc) reaching top_p.  Order
//      by p equals order by f, so the cut is found by a radix select on the
//      orderable 32-bit key of f with fp64 mass histograms, 12 + 10 + 10 bits
//      (a first pass on the top 8 bits would put a row of N(0,1)-like logits
//      into a handful of sign/exponent buckets and serialise the LDS
//      atomics).  The crossing bucket is found by a block suffix scan.  The
//      select yields the threshold key T, the mass of keys above T, and how
//      many of the elements tied at T (in id order) complete the nucleus.
//   3. u = top 24 bits of word 0 of Philox4x32-10 (key = seed halves,
//      counter = (row in session, session, 0, 0)) times 2^-24; the token is
//      the first nucleus member in ascending id order whose running mass
//      exceeds u * mass(nucleus) (the last member if rounding leaves none).
//
// The weights are recomputed in fp64 in every pass instead of stored: a row
// of 65536 fp64 weights does not fit the registers of a 1024-thread block,
// and fp32 weights would move the nucleus cut by ~1e-8 of the row's mass.
// Histogram bins are accumulated with LDS fp64 atomics; their order can
// change the last bit of a bin, which matters only for rows whose cut lies
// within ~1e-16 of a bin boundary.
#include "sph_internal.h"

namespace sph {

constexpr int kSampleThreads = 1024;
constexpr int kSampleWaves = kSampleThreads / 64;

__device__ __forceinline__ uint32_t orderable(float v) {
  v = v + 0.0f;
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_orderable(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
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

__device__ __forceinline__ double shfl_xor_f64(double x, int o) {
  const unsigned long long b = __double_as_longlong(x);
  const uint32_t lo = __shfl_xor((uint32_t)b, o, 64);
  const uint32_t hi = __shfl_xor((uint32_t)(b >> 32), o, 64);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

__device__ __forceinline__ double shfl_up_f64(double x, int o) {
  const unsigned long long b = __double_as_longlong(x);
  const uint32_t lo = __shfl_up((uint32_t)b, o, 64);
  const uint32_t hi = __shfl_up((uint32_t)(b >> 32), o, 64);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

constexpr int kRadixBuckets = 4096;  // widest pass: 12 bits
constexpr int kBucketsPerThread = kRadixBuckets / kSampleThreads;

struct SampleShared {
  double hist[kRadixBuckets];
  uint32_t cnt[kRadixBuckets];
  double wred[kSampleWaves];
  uint32_t ured[kSampleWaves];
  float fred[kSampleWaves];
  uint32_t bc_u[2];
  int32_t pick;
  int32_t last;
};

// Block-wide reductions and scans in a fixed order (deterministic).
__device__ float block_max_f32(float v, SampleShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  __syncthreads();
  if (lane == 0) sh.fred[wave] = v;
  __syncthreads();
  float r = sh.fred[0];
  for (int w = 1; w < kSampleWaves; ++w) r = fmaxf(r, sh.fred[w]);
  return r;
}

__device__ double block_sum_f64(double v, SampleShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += shfl_xor_f64(v, o);
  __syncthreads();
  if (lane == 0) sh.wred[wave] = v;
  __syncthreads();
  double r = 0.0;
  for (int w = 0; w < kSampleWaves; ++w) r += sh.wred[w];
  return r;
}

// Exclusive prefix sum over threads (thread order = id order); *total = sum.
__device__ double block_exscan_f64(double v, SampleShared& sh, double* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y = shfl_up_f64(inc, o);
    if (lane >= o) inc += y;
  }
  __syncthreads();
  if (lane == 63) sh.wred[wave] = inc;
  __syncthreads();
  double base = 0.0, tot = 0.0;
  for (int w = 0; w < kSampleWaves; ++w) {
    if (w < wave) base += sh.wred[w];
    tot += sh.wred[w];
  }
  *total = tot;
  return base + inc - v;
}

__device__ uint32_t block_exscan_u32(uint32_t v, SampleShared& sh, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  __syncthreads();
  if (lane == 63) sh.ured[wave] = inc;
  __syncthreads();
  uint32_t base = 0, tot = 0;
  for (int w = 0; w < kSampleWaves; ++w) {
    if (w < wave) base += sh.ured[w];
    tot += sh.ured[w];
  }
  *total = tot;
  return base + inc - v;
}

// Apply fn(i) to the thread's elements i = 0 .. cnt-1 in id order.  With
// CH > 0 the loop is unrolled so register-held values are indexed statically.
template <int CH, class F>
__device__ __forceinline__ void for_each_elem(int cnt, F&& fn) {
  if constexpr (CH > 0) {
#pragma unroll
    for (int i = 0; i < CH; ++i)
      if (i < cnt) fn(i);
  } else {
    for (int i = 0; i < cnt; ++i) fn(i);
  }
}

// CH > 0: the thread's CH values live in registers (n <= 1024 * CH).
// CH == 0: values are re-read from f in every pass (any n).
template <int CH>
__global__ __launch_bounds__(kSampleThreads) void k_sample(const float* __restrict__ f, int n,
                                                           const int32_t* __restrict__ ids, int R,
                                                           float temperature, float top_p,
                                                           uint32_t seed_lo, uint32_t seed_hi,
                                                           int32_t* __restrict__ tokens) {
  __shared__ SampleShared sh;
  const int m = blockIdx.x;
  const int t = threadIdx.x;
  const float* row = f + (int64_t)m * n;
  const int ch = CH > 0 ? CH : (n + kSampleThreads - 1) / kSampleThreads;
  const int p0 = t * ch;
  const int cnt = max(0, min(n, p0 + ch) - p0);

  float vreg[CH > 0 ? CH : 1];
  if constexpr (CH > 0) {
#pragma unroll
    for (int i = 0; i < CH; ++i) vreg[i] = i < cnt ? row[p0 + i] : 0.0f;
  }
  auto val = [&](int i) -> float {
    if constexpr (CH > 0) return vreg[i];
    else return row[p0 + i];
  };

  // 1. max and partition function
  float lmax = -INFINITY;
  for_each_elem<CH>(cnt, [&](int i) { lmax = fmaxf(lmax, val(i)); });
  const float fmax = block_max_f32(lmax, sh);
  const double tau = (double)temperature;
  const double dmax = (double)fmax;
  auto weight = [&](float x) -> double { return exp(((double)x - dmax) / tau); };
  double lsum = 0.0;
  for_each_elem<CH>(cnt, [&](int i) { lsum += weight(val(i)); });
  const double Z = block_sum_f64(lsum, sh);

  // 2. nucleus threshold by radix select on the orderable key
  const double tp = (double)top_p;
  uint32_t T = 0u, mask = 0u;
  double above = 0.0;  // mass of the elements whose key lies above the current prefix
  uint32_t c_ties = 0u;
  const bool all = tp >= 1.0;
  if (!all) {
    const double need = tp * Z;
    constexpr int kShift[3] = {20, 10, 0};
    constexpr int kBits[3] = {12, 10, 10};
#pragma unroll
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = kShift[pass], nb = 1 << kBits[pass];
      for (int b = t; b < nb; b += kSampleThreads) {
        sh.hist[b] = 0.0;
        sh.cnt[b] = 0u;
      }
      if (t == 0) {
        sh.bc_u[0] = 0xFFFFFFFFu;
        sh.bc_u[1] = 0xFFFFFFFFu;
      }
      __syncthreads();
      for_each_elem<CH>(cnt, [&](int i) {
        const float x = val(i);
        const uint32_t k = orderable(x);
        if ((k & mask) == T) {
          const int b = (k >> shift) & (nb - 1);
          atomicAdd(&sh.hist[b], weight(x));
          atomicAdd(&sh.cnt[b], 1u);
        }
      });
      __syncthreads();
      // Thread t owns buckets nb-1-(kBucketsPerThread*t + i): descending keys.
      double local[kBucketsPerThread];
      double lsb = 0.0;
#pragma unroll
      for (int i = 0; i < kBucketsPerThread; ++i) {
        const int b = nb - 1 - (kBucketsPerThread * t + i);
        local[i] = b >= 0 ? sh.hist[b] : 0.0;
        lsb += local[i];
      }
      double tot = 0.0;
      double acc = above + block_exscan_f64(lsb, sh, &tot);
      bool crossed = false;
#pragma unroll
      for (int i = 0; i < kBucketsPerThread; ++i) {
        const int b = nb - 1 - (kBucketsPerThread * t + i);
        if (b >= 0 && !crossed && sh.cnt[b] != 0u) {
          if (acc + local[i] >= need) {
            atomicMin(&sh.bc_u[0], (uint32_t)(nb - 1 - b));  // the highest crossing bucket
            crossed = true;
          }
        }
        acc += local[i];
      }
#pragma unroll
      for (int i = kBucketsPerThread - 1; i >= 0; --i) {  // lowest non-empty bucket
        const int b = nb - 1 - (kBucketsPerThread * t + i);
        if (b >= 0 && sh.cnt[b] != 0u) {
          atomicMin(&sh.bc_u[1], (uint32_t)b);
          break;
        }
      }
      __syncthreads();
      // A target that rounding left above the range's total takes everything.
      const uint32_t sel =
          sh.bc_u[0] != 0xFFFFFFFFu ? (uint32_t)(nb - 1) - sh.bc_u[0] : sh.bc_u[1];
      double part = 0.0;
#pragma unroll
      for (int i = 0; i < kBucketsPerThread; ++i) {
        const int b = nb - 1 - (kBucketsPerThread * t + i);
        if (b > (int)sel) part += local[i];
      }
      above += block_sum_f64(part, sh);
      T |= sel << shift;
      mask |= (uint32_t)(nb - 1) << shift;
      if (pass == 2) {
        // smallest c in [1, ties] with above + c * e_T >= need
        const uint32_t nt = sh.cnt[sel];
        const double eT = weight(from_orderable(T));
        double cd = ceil((need - above) / eT);
        uint32_t c = cd < 1.0 ? 1u : (cd > (double)nt ? nt : (uint32_t)cd);
        while (c > 1u && above + (double)(c - 1u) * eT >= need) --c;
        while (c < nt && above + (double)c * eT < need) ++c;
        c_ties = c;
      }
      __syncthreads();
    }
  }

  // tie ranks in id order, then member masses in id order
  uint32_t my_ties = 0u;
  if (!all) for_each_elem<CH>(cnt, [&](int i) { my_ties += orderable(val(i)) == T ? 1u : 0u; });
  uint32_t tie_tot = 0u;
  const uint32_t tie_base = block_exscan_u32(my_ties, sh, &tie_tot);
  auto is_member = [&](float x, uint32_t& tie_seen) -> bool {
    if (all) return true;
    const uint32_t k = orderable(x);
    if (k > T) return true;
    if (k == T) return tie_base + tie_seen++ < c_ties;
    return false;
  };
  double my_mass = 0.0;
  int my_last = -1;
  {
    uint32_t ts = 0u;
    for_each_elem<CH>(cnt, [&](int i) {
      const float x = val(i);
      if (is_member(x, ts)) {
        my_mass += weight(x);
        my_last = p0 + i;
      }
    });
  }
  double mass = 0.0;
  const double base = block_exscan_f64(my_mass, sh, &mass);

  // 3. inverse CDF in ascending id order
  const uint32_t s_idx = (uint32_t)(m / R), r_idx = (uint32_t)(m % R);
  const uint32_t x0 = philox_x0(r_idx, s_idx, 0u, 0u, seed_lo, seed_hi);
  const double target = (double)(x0 >> 8) * 0x1.0p-24 * mass;
  if (t == 0) {
    sh.pick = 0x7FFFFFFF;
    sh.last = -1;
  }
  __syncthreads();
  if (my_mass > 0.0 && base <= target && target < base + my_mass) {
    // The claimed interval comes from a scan whose rounding can differ from
    // this walk's by an ulp; the walk falls back to its own last member.
    double run = base;
    uint32_t ts = 0u;
    int pos = my_last;
    bool found = false;
    for_each_elem<CH>(cnt, [&](int i) {
      const float x = val(i);
      if (is_member(x, ts) && !found) {
        run += weight(x);
        if (run > target) {
          pos = p0 + i;
          found = true;
        }
      }
    });
    atomicMin(&sh.pick, pos);
  }
  if (my_last >= 0) atomicMax(&sh.last, my_last);
  __syncthreads();
  if (t == 0) {
    const int pos = sh.pick != 0x7FFFFFFF ? sh.pick : sh.last;
    tokens[m] = ids[pos >= 0 ? pos : 0];
  }
}

__global__ void k_accept(const int32_t* __restrict__ tokens, const int32_t* __restrict__ drafts,
                         int n_sessions, int R, int32_t* __restrict__ accept) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_sessions) return;
  const int kd = R - 1;
  int a = 0;
  while (a < kd && tokens[(int64_t)s * R + a] == drafts[(int64_t)s * kd + a]) ++a;
  accept[s] = a;
}

hipError_t launch_sample(const float* f, int M, int n, const int32_t* ids, int R,
                         float temperature, float top_p, uint64_t seed, int32_t* tokens,
                         hipStream_t s) {
  const uint32_t lo = (uint32_t)seed, hi = (uint32_t)(seed >> 32);
  if (n <= kSampleThreads * 16)
    hipLaunchKernelGGL(k_sample<16>, dim3(M), dim3(kSampleThreads), 0, s, f, n, ids, R,
                       temperature, top_p, lo, hi, tokens);
  else if (n <= kSampleThreads * 64)
    hipLaunchKernelGGL(k_sample<64>, dim3(M), dim3(kSampleThreads), 0, s, f, n, ids, R,
                       temperature, top_p, lo, hi, tokens);
  else
    hipLaunchKernelGGL(k_sample<0>, dim3(M), dim3(kSampleThreads), 0, s, f, n, ids, R,
                       temperature, top_p, lo, hi, tokens);
  return hipGetLastError();
}

hipError_t launch_accept(const int32_t* tokens, const int32_t* drafts, int n_sessions, int R,
                         int32_t* accept, hipStream_t s) {
  hipLaunchKernelGGL(k_accept, dim3((n_sessions + 255) / 256), dim3(256), 0, s, tokens, drafts,
                     n_sessions, R, accept);
  return hipGetLastError();
}

}  // namespace sph
