// Row-wide epilogues that need a whole row: the int8 payload quantiser and
// the greedy finaliser with draft verification.
#include "sph_internal.h"

namespace sph {

constexpr int kQuantChunk = 4096;  // columns per quantiser block (256 threads x 16)

// One b-bit code (qmax = 2^(b-1) - 1) of z with scale s.
__device__ __forceinline__ int quantize_one(float z, float clip, float s, float qmax) {
  const float y = fminf(fmaxf(z, -clip), clip);
  // s == 0 only for a row or block that is exactly zero after the clip.
  const float t = s > 0.0f ? y / s : 0.0f;
  return (int)fminf(fmaxf(rintf(t), -qmax), qmax);
}

// Clip + symmetric b-bit quantisation (Section 5.4 "after clipping,
// quantization"; eq. 18 with a configurable bit width b).  Grid (rows, column
// chunks of 4096).  With one scale per row (qshift < 0) every block first
// folds the row's per-block maxima of |clamp(z)| (written by the projection)
// into a_m, so all blocks of a row agree on s = a_m / qmax bit for bit.  With
// one scale per block of 2^qshift positions (256 ... 4096, so a block never
// straddles a chunk) the chunk's blocks take their maxima from z itself.
// The division is correctly rounded.  8-bit codes are bytes; 4-bit codes go
// two per byte, the even position in the low nibble (two's complement).
template <int BITS>
__global__ __launch_bounds__(256) void k_quantize(const float* __restrict__ z,
                                                  const float* __restrict__ amax_part, int nblk,
                                                  int n, int vec, float clip, int qshift,
                                                  uint8_t* __restrict__ q, int64_t qstride,
                                                  float* __restrict__ scale, int qnb) {
  constexpr float kQmax = BITS == 8 ? 127.0f : 7.0f;
  const int m = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ float s_red[4];
  __shared__ uint32_t s_bmax[kQuantChunk / 256];  // |y| maxima of the chunk's blocks
  const int64_t zrow = (int64_t)m * n;
  const int j0 = blockIdx.y * kQuantChunk;
  const int j1 = min(n, j0 + kQuantChunk);
  const bool per_row = qshift < 0;

  // the chunk's z values of this thread (4 consecutive columns per 1024), all
  // loaded before any is used, and before the row's partial maxima, so the
  // two loads' latencies overlap
  constexpr int VT = kQuantChunk / 1024;
  float4 v[VT];
#pragma unroll
  for (int t = 0; t < VT; ++t) {
    const int j = j0 + tid * 4 + 1024 * t;
    if (vec) {
      v[t] = j < j1 ? *reinterpret_cast<const float4*>(z + zrow + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
      v[t].x = j < j1 ? z[zrow + j] : 0.f;
      v[t].y = j + 1 < j1 ? z[zrow + j + 1] : 0.f;
      v[t].z = j + 2 < j1 ? z[zrow + j + 2] : 0.f;
      v[t].w = j + 3 < j1 ? z[zrow + j + 3] : 0.f;
    }
  }
  float srow = 0.0f;
  if (per_row) {
    // all of a thread's partial maxima are loaded at once (no load waits on
    // the previous one)
    constexpr int PT = kMaxBlocks / 256;
    float part[PT];
#pragma unroll
    for (int t = 0; t < PT; ++t) {
      const int i = tid + 256 * t;
      part[t] = i < nblk ? amax_part[(int64_t)m * kMaxBlocks + i] : 0.0f;
    }
    float a = 0.0f;
#pragma unroll
    for (int t = 0; t < PT; ++t) a = fmaxf(a, part[t]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) a = fmaxf(a, __shfl_xor(a, o, 64));
    if (lane == 0) s_red[wave] = a;
    __syncthreads();
    a = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
    srow = a / kQmax;
    if (blockIdx.y == 0 && tid == 0) scale[(int64_t)m * qnb] = srow;
  } else if (tid < kQuantChunk / 256) {
    s_bmax[tid] = 0u;
  }

  auto absclip = [&](float x) { return fabsf(fminf(fmaxf(x, -clip), clip)); };
  if (!per_row) {
    // a wave's 256 columns of one iteration lie in one block
    __syncthreads();
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      float a = fmaxf(fmaxf(absclip(v[t].x), absclip(v[t].y)), fmaxf(absclip(v[t].z), absclip(v[t].w)));
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) a = fmaxf(a, __shfl_xor(a, o, 64));
      const int j = j0 + 1024 * t + 256 * wave;
      if (lane == 0 && j < j1) atomicMax(&s_bmax[(j - j0) >> qshift], __float_as_uint(a));
    }
    __syncthreads();
    const int nbk = ((j1 - j0) + (1 << qshift) - 1) >> qshift;
    if (tid < nbk) scale[(int64_t)m * qnb + (j0 >> qshift) + tid] = __uint_as_float(s_bmax[tid]) / kQmax;
  }

  uint8_t* qrow = q + (int64_t)m * qstride;
#pragma unroll
  for (int t = 0; t < VT; ++t) {
    const int j = j0 + tid * 4 + 1024 * t;
    if (j >= j1) continue;
    const float s = per_row ? srow : __uint_as_float(s_bmax[(j - j0) >> qshift]) / kQmax;
    const int c0 = quantize_one(v[t].x, clip, s, kQmax), c1 = quantize_one(v[t].y, clip, s, kQmax);
    const int c2 = quantize_one(v[t].z, clip, s, kQmax), c3 = quantize_one(v[t].w, clip, s, kQmax);
    if constexpr (BITS == 8) {
      if (vec) {
        char4 o;
        o.x = (signed char)c0;
        o.y = (signed char)c1;
        o.z = (signed char)c2;
        o.w = (signed char)c3;
        *reinterpret_cast<char4*>(qrow + j) = o;
      } else {
        const int c[4] = {c0, c1, c2, c3};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (j + e < j1) qrow[j + e] = (uint8_t)(int8_t)c[e];
      }
    } else {
      // columns past the row quantise to 0 (their z is 0), which is the pad
      // nibble of an odd row
      const uint8_t b0 = (uint8_t)((c0 & 15) | ((c1 & 15) << 4));
      const uint8_t b1 = (uint8_t)((c2 & 15) | ((c3 & 15) << 4));
      qrow[j >> 1] = b0;
      if (j + 2 < j1) qrow[(j >> 1) + 1] = b1;
    }
  }
}

hipError_t launch_quantize(const float* z, const float* amax_part, int nblk, int M, int n,
                           float clip, int bits, int qshift, uint8_t* q, int64_t qstride,
                           float* scale, int qnb, hipStream_t s) {
  const int chunks = (n + kQuantChunk - 1) / kQuantChunk;
  if (chunks > 65535 || (bits != 8 && bits != 4)) return hipErrorInvalidValue;
  if (qshift >= 0 && (qshift < 8 || (1 << qshift) > kQuantChunk)) return hipErrorInvalidValue;
  // float4 / char4 accesses need whole, aligned groups of four columns
  const int vec = (n % 4 == 0) && (reinterpret_cast<uintptr_t>(z) % 16 == 0) &&
                  (reinterpret_cast<uintptr_t>(q) % 4 == 0) && qstride % 4 == 0;
  if (bits == 8)
    launch_kernel(k_quantize<8>, dim3(M, chunks), dim3(256), 0, s, z, amax_part, nblk, n, vec,
                  clip, qshift, q, qstride, scale, qnb);
  else
    launch_kernel(k_quantize<4>, dim3(M, chunks), dim3(256), 0, s, z, amax_part, nblk, n, vec,
                  clip, qshift, q, qstride, scale, qnb);
  return hipGetLastError();
}

__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long x, int o) {
  const uint32_t lo = __shfl_xor((uint32_t)x, o, 64);
  const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), o, 64);
  return ((unsigned long long)hi << 32) | lo;
}

constexpr int kMaxRowsPerSession = 1024;
constexpr int kFinalWaves = 16;  // rows of a session reduced in parallel

// One block per session, one wave per verification row: fold the row's
// per-block argmax keys (every lane loads its share of up to kMaxBlocks keys
// at once) into the greedy token, ties to the lowest subset position = the
// lowest id; then count the drafts that match the verification rows in
// order (Section 5.5, Algorithm 1 verification step).
__global__ __launch_bounds__(64 * kFinalWaves) void k_final_greedy(
    const unsigned long long* __restrict__ best, int nblk, const int32_t* __restrict__ ids, int n,
    int R, const int32_t* __restrict__ drafts, int32_t* __restrict__ tokens,
    int32_t* __restrict__ accept) {
  constexpr int PER_LANE = kMaxBlocks / 64;
  const int s = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ int32_t s_tok[kMaxRowsPerSession];
  __shared__ int32_t s_draft[kMaxRowsPerSession];
  // the session's drafts are staged while the keys are read, so the prefix
  // match below reads LDS only
  for (int r = tid; r < R - 1; r += blockDim.x) s_draft[r] = drafts[(int64_t)s * (R - 1) + r];
  for (int r = wave; r < R; r += kFinalWaves) {
    const int64_t m = (int64_t)s * R + r;
    unsigned long long x[PER_LANE];
#pragma unroll
    for (int t = 0; t < PER_LANE; ++t) {
      const int i = lane + 64 * t;
      x[t] = i < nblk ? best[m * kMaxBlocks + i] : 0ull;
    }
    unsigned long long k = x[0];
#pragma unroll
    for (int t = 1; t < PER_LANE; ++t) k = x[t] > k ? x[t] : k;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const unsigned long long y = shfl_xor_u64(k, o);
      k = y > k ? y : k;
    }
    if (lane == 0) {
      // every position of the row produced a key, so pos < n; the clamp only
      // keeps a corrupted key from reading outside the id table
      const uint32_t pos = min(0xFFFFFFFFu - (uint32_t)k, (uint32_t)(n - 1));
      const int32_t tok = ids[pos];
      tokens[m] = tok;
      s_tok[r] = tok;
    }
  }
  __syncthreads();
  if (tid == 0) {
    const int kd = R - 1;
    int a = 0;
    while (a < kd && s_tok[a] == s_draft[a]) ++a;
    accept[s] = a;
  }
}

hipError_t launch_final_greedy(const uint64_t* best_part, int nblk, const int32_t* ids, int n,
                               int n_sessions, int R, const int32_t* drafts, int32_t* tokens,
                               int32_t* accept, hipStream_t s) {
  if (R > kMaxRowsPerSession || n < 1 || nblk > kMaxBlocks) return hipErrorInvalidValue;
  const int waves = R < kFinalWaves ? R : kFinalWaves;
  launch_kernel(k_final_greedy, dim3(n_sessions), dim3(64 * waves), 0, s,
                     reinterpret_cast<const unsigned long long*>(best_part), nblk, ids, n, R,
                     drafts, tokens, accept);
  return hipGetLastError();
}

}  // namespace sph
