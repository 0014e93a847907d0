// Hidden-state codes: the cloud quantises the hidden state it returns
// (Section 5.3: every returned tensor is quantised with the Q_b of eq. 18,
// here b = 8 with one scale per row), and the endpoint widens the codes into
// bf16 operands for its projection (eq. 11 on the dequantised values).
#include "sph_internal.h"

namespace sph {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kHqThreads = 256;
constexpr int kHqVecPerThread = 4;  // 16-byte chunks a thread keeps in registers
constexpr int kHqRegCols = kHqThreads * kHqVecPerThread * 8;  // 8192 columns

__device__ __forceinline__ float bf16_value(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// One int8 code of x with scale s: rint(x / s) (correctly rounded division,
// ties to even) clamped to +-127; 0 for s == 0, which only a zero row has.
__device__ __forceinline__ int hidden_code(float x, float s) {
  const float t = s > 0.0f ? x / s : 0.0f;
  return (int)fminf(fmaxf(rintf(t), -127.0f), 127.0f);
}

__device__ __forceinline__ float block_max(float a, float* s_red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) a = fmaxf(a, __shfl_xor(a, o, 64));
  if (lane == 0) s_red[wave] = a;
  __syncthreads();
  return fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
}

// One block per row.  VEC: the row is 16-byte aligned, d is a multiple of 8
// and at most 8192, so each thread loads its chunks once, keeps them in
// registers for both the maximum and the codes, and stores 8 codes at a
// time.  Otherwise the row is read twice (the second time from cache).
template <bool VEC>
__global__ __launch_bounds__(kHqThreads) void k_hidden_quantize(const uint16_t* __restrict__ h,
                                                                int64_t ldh, int d,
                                                                int8_t* __restrict__ q,
                                                                int64_t ldq,
                                                                float* __restrict__ scale) {
  __shared__ float s_red[kHqThreads / 64];
  const int64_t m = blockIdx.x;
  const int tid = threadIdx.x;
  const uint16_t* row = h + m * ldh;
  int8_t* qrow = q + m * ldq;
  if constexpr (VEC) {
    u32x4_t v[kHqVecPerThread];
    float a = 0.0f;
#pragma unroll
    for (int t = 0; t < kHqVecPerThread; ++t) {
      const int c = (tid + t * kHqThreads) * 8;
      v[t] = c < d ? *reinterpret_cast<const u32x4_t*>(row + c) : u32x4_t{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int t = 0; t < kHqVecPerThread; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a = fmaxf(a, fabsf(bf16_value(v[t][e] & 0xFFFFu)));
        a = fmaxf(a, fabsf(bf16_value(v[t][e] >> 16)));
      }
    const float s = block_max(a, s_red) / 127.0f;
    if (tid == 0) scale[m] = s;
#pragma unroll
    for (int t = 0; t < kHqVecPerThread; ++t) {
      const int c = (tid + t * kHqThreads) * 8;
      if (c >= d) continue;
      uint32_t w[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo = (uint32_t)(hidden_code(bf16_value(v[t][e] & 0xFFFFu), s) & 0xFF);
        const uint32_t hi = (uint32_t)(hidden_code(bf16_value(v[t][e] >> 16), s) & 0xFF);
        w[e >> 1] |= (lo | (hi << 8)) << (16 * (e & 1));
      }
      if ((reinterpret_cast<uintptr_t>(qrow + c) & 7) == 0) {
        *reinterpret_cast<uint2*>(qrow + c) = make_uint2(w[0], w[1]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qrow[c + e] = (int8_t)(w[e >> 2] >> (8 * (e & 3)));
      }
    }
  } else {
    float a = 0.0f;
    for (int k = tid; k < d; k += kHqThreads) a = fmaxf(a, fabsf(bf16_value(row[k])));
    const float s = block_max(a, s_red) / 127.0f;
    if (tid == 0) scale[m] = s;
    for (int k = tid; k < d; k += kHqThreads) qrow[k] = (int8_t)hidden_code(bf16_value(row[k]), s);
  }
}

hipError_t launch_hidden_quantize(const uint16_t* h, int64_t ldh, int M, int d, int8_t* q,
                                  int64_t ldq, float* scale, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const bool vec = d % 8 == 0 && d <= kHqRegCols && ldh % 8 == 0 &&
                   (reinterpret_cast<uintptr_t>(h) & 15) == 0;
  if (vec)
    launch_kernel(k_hidden_quantize<true>, dim3(M), dim3(kHqThreads), 0, s, h, ldh, d, q, ldq, scale);
  else
    launch_kernel(k_hidden_quantize<false>, dim3(M), dim3(kHqThreads), 0, s, h, ldh, d, q, ldq, scale);
  return hipGetLastError();
}

// Codes -> bf16 operands: every int8 value has at most 8 significant bits,
// so (float)code truncated to its upper 16 bits is exact.  out is [M, Kp]
// (Kp = K rounded up to 8, the pad columns zero); one thread per 8 columns.
__global__ __launch_bounds__(256) void k_widen_codes(const int8_t* __restrict__ hq, int64_t ldhq,
                                                     int K, int Kp, int64_t groups,
                                                     uint16_t* __restrict__ out) {
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (g >= groups) return;
  const int gpr = Kp / 8;
  const int64_t m = g / gpr;
  const int c = (int)(g - m * gpr) * 8;
  const int8_t* src = hq + m * ldhq;
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int k0 = c + 2 * e;
    const uint32_t lo = k0 < K ? __float_as_uint((float)src[k0]) >> 16 : 0u;
    const uint32_t hi = k0 + 1 < K ? __float_as_uint((float)src[k0 + 1]) >> 16 : 0u;
    w[e] = lo | (hi << 16);
  }
  *reinterpret_cast<u32x4_t*>(out + m * Kp + c) = u32x4_t{w[0], w[1], w[2], w[3]};
}

hipError_t launch_widen_codes(const int8_t* hq, int64_t ldhq, int M, int K, int Kp,
                              uint16_t* out, hipStream_t s) {
  if (M <= 0 || Kp <= 0) return hipSuccess;
  if (Kp % 8 != 0 || Kp < K) return hipErrorInvalidValue;
  const int64_t groups = (int64_t)M * (Kp / 8);
  const int64_t blocks = (groups + 255) / 256;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  launch_kernel(k_widen_codes, dim3((unsigned)blocks), dim3(256), 0, s, hq, ldhq, K, Kp, groups, out);
  return hipGetLastError();
}

}  // namespace sph
