// Row-wide epilogues that need a whole row: the int8 payload quantiser and
// the greedy finaliser with draft verification.
#include "sph_internal.h"

namespace sph {

constexpr int kQuantChunk = 4096;  // columns per quantiser block (256 threads x 16)

__device__ __forceinline__ int8_t quantize_one(float z, float clip, float s) {
  const float y = fminf(fmaxf(z, -clip), clip);
  // s == 0 only for a row that is exactly zero after the clip.
  const float t = s > 0.0f ? y / s : 0.0f;
  const float r = fminf(fmaxf(rintf(t), -127.0f), 127.0f);
  return (int8_t)(int)r;
}

// Clip + per-row symmetric int8 (Section 5.4 "after clipping, quantization";
// eq. 18 with b = 8).  Every block first folds
// the row's per-block maxima of |clamp(z)| (written by the projection) into
// a_m, then derives s = a_m / 127 with a correctly rounded division, so all
// blocks of a row agree on s bit for bit.  Grid (rows, column chunks).
__global__ __launch_bounds__(256) void k_quantize(const float* __restrict__ z,
                                                  const float* __restrict__ amax_part, int nblk,
                                                  int n, int vec, float clip,
                                                  int8_t* __restrict__ q,
                                                  float* __restrict__ scale) {
  const int m = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ float s_red[4];
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
  const float s = a / 127.0f;
  if (blockIdx.y == 0 && tid == 0) scale[m] = s;

  const int64_t row = (int64_t)m * n;
  const int j0 = blockIdx.y * kQuantChunk;
  const int j1 = min(n, j0 + kQuantChunk);
  if (vec) {
    // the chunk's z values of this thread are loaded before any is stored
    constexpr int VT = kQuantChunk / 1024;
    float4 v[VT];
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      const int j = j0 + tid * 4 + 1024 * t;
      v[t] = j < j1 ? *reinterpret_cast<const float4*>(z + row + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int t = 0; t < VT; ++t) {
      const int j = j0 + tid * 4 + 1024 * t;
      if (j >= j1) continue;
      char4 o;
      o.x = quantize_one(v[t].x, clip, s);
      o.y = quantize_one(v[t].y, clip, s);
      o.z = quantize_one(v[t].z, clip, s);
      o.w = quantize_one(v[t].w, clip, s);
      *reinterpret_cast<char4*>(q + row + j) = o;
    }
  } else {
    for (int j = j0 + tid; j < j1; j += 256) q[row + j] = quantize_one(z[row + j], clip, s);
  }
}

hipError_t launch_quantize(const float* z, const float* amax_part, int nblk, int M, int n,
                           float clip, int8_t* q, float* scale, hipStream_t s) {
  const int chunks = (n + kQuantChunk - 1) / kQuantChunk;
  if (chunks > 65535) return hipErrorInvalidValue;
  // float4 / char4 accesses need whole, aligned groups of four columns
  const int vec = (n % 4 == 0) && (reinterpret_cast<uintptr_t>(z) % 16 == 0) &&
                  (reinterpret_cast<uintptr_t>(q) % 4 == 0);
  launch_kernel(k_quantize, dim3(M, chunks), dim3(256), 0, s, z, amax_part, nblk, n, vec,
                     clip, q, scale);
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
