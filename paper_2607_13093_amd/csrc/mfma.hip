// Dense gathered projection for many rows of h (MFMA path).
//
//   C[m, j] = sum_k h[m, k] * W[S_j, k]      (eq. 12 / eq. 11 on the subset S)
//
// With hundreds of rows the contraction is dense enough for the matrix
// cores: a block computes a BM x BN tile of C with v_mfma_f32_32x32x16_bf16
// (bf16 inputs, fp32 accumulation).  Both operands are K-contiguous in
// memory (h is [M, K] row-major, the weight rows are vocab-major), so both
// tiles are staged in LDS as [rows][BK] with a 16-byte row pad, which makes
// every operand fetch a conflict-free ds_read_b128.  The B tile is gathered:
// tile column j is weight row S[n0 + j]; fp8 E4M3 rows are widened to bf16
// (exactly) on their way into LDS and their per-row scale is applied in the
// epilogue.  Global loads of the next K step are issued into registers
// before the MFMAs of the current step.
//
// Operand layouts of the 32x32x16 instruction (checked on the hardware):
//   A: lane l supplies A[l % 32][8 * (l / 32) + e], e = 0..7
//   B: lane l supplies B[8 * (l / 32) + e][l % 32]
//   C: accumulator r of lane l is C[8 * (r / 4) + 4 * (l / 32) + r % 4][l % 32]
//
// Tile order: blocks are dealt round-robin to the 8 XCDs, so block b is
// remapped to give each XCD a contiguous range of tiles, and tiles are
// numbered with the m-tiles of one n-tile adjacent (groups of up to GM):
// blocks sharing a gathered B tile (or an A panel) run on the same XCD at the
// same time and meet in its L2.
//
// Epilogues: the cloud epilogue scales fp8 columns, adds the bias, writes
// fp32 partial logits and the tile's row maxima of |clamp(z)|; the fuse
// epilogue dequantises the payload (eq. 13), writes fused logits on request
// and the tile's per-row (value, position) argmax key.
#include "sph_internal.h"

namespace sph {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_to_bf16x2_m(uint32_t x) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, HI));
}

__device__ __forceinline__ unsigned long long argmax_key_m(float v, int pos) {
  v = v + 0.0f;  // -0 -> +0
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)u << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)pos);
}

__device__ __forceinline__ unsigned long long shfl_xor_u64_m(unsigned long long x, int o) {
  const uint32_t lo = __shfl_xor((uint32_t)x, o, 64);
  const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), o, 64);
  return ((unsigned long long)hi << 32) | lo;
}

constexpr int kBK = 64;          // K elements per staged step
constexpr int kLDK = kBK + 8;    // padded LDS row, bf16 elements (144 bytes)
constexpr int kGM = 4;           // m-tiles grouped per n-tile in the tile order

__device__ __forceinline__ void tile_of_block(int b, int m_tiles, int n_tiles, int& mt, int& nt) {
  const int total = m_tiles * n_tiles;
  const int full = total / 8 * 8;
  const int tile = b < full ? (b % 8) * (full / 8) + b / 8 : b;
  const int gm_max = m_tiles < kGM ? m_tiles : kGM;
  const int group = gm_max * n_tiles;
  const int g = tile / group;
  const int first_m = g * gm_max;
  const int gm = min(m_tiles - first_m, gm_max);
  const int in = tile - g * group;
  mt = first_m + in % gm;
  nt = in / gm;
}

template <int BM, int BN, int WM, int WN, int WT, int EPI>
__global__ __launch_bounds__(64 * WM * WN) void k_mfma(const MfmaArgs a) {
  constexpr int NT = 64 * WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;  // wave tile
  constexpr int FM = TM / 32, FN = TN / 32;  // 32x32 fragments per wave
  constexpr int A_CH = BM * (kBK / 8) / NT;  // 16-byte A chunks per thread
  constexpr int B_EPC = WT == 0 ? 8 : 16;    // weight elements per 16-byte chunk
  constexpr int B_CH = BN * (kBK / B_EPC) / NT;
  static_assert(A_CH * NT == BM * (kBK / 8) && B_CH * NT == BN * (kBK / B_EPC), "tile/threads");

  __shared__ __align__(16) uint16_t As[BM * kLDK];
  __shared__ __align__(16) uint16_t Bs[BN * kLDK];
  __shared__ int32_t s_ids[BN];
  __shared__ uint32_t s_rmax[BM];
  __shared__ unsigned long long s_rkey[BM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  int mt, nt;
  tile_of_block(blockIdx.x, a.m_tiles, a.n_tiles, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int M = a.M, K = a.K, n = a.n;

  for (int i = tid; i < BN; i += NT) s_ids[i] = n0 + i < n ? a.ids[n0 + i] : -1;
  for (int i = tid; i < BM; i += NT) {
    s_rmax[i] = 0u;
    s_rkey[i] = 0ull;
  }
  __syncthreads();

  u32x4_t ra[A_CH], rb[B_CH];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + i * NT, row = c >> 3, kk = k0 + (c & 7) * 8;
      const int gr = m0 + row;
      ra[i] = (gr < M && kk < K) ? *reinterpret_cast<const u32x4_t*>(a.h + (int64_t)gr * a.ldh + kk)
                                 : u32x4_t{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + i * NT;
      const int row = c / (kBK / B_EPC), kk = k0 + (c % (kBK / B_EPC)) * B_EPC;
      const int id = s_ids[row];
      rb[i] = (id >= 0 && kk < K)
                  ? __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(
                        a.w + (int64_t)id * a.ldw_bytes + (int64_t)kk * (WT == 0 ? 2 : 1)))
                  : u32x4_t{0u, 0u, 0u, 0u};
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + i * NT, row = c >> 3, kc = c & 7;
      *reinterpret_cast<u32x4_t*>(As + row * kLDK + kc * 8) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + i * NT;
      const int row = c / (kBK / B_EPC), kc = c % (kBK / B_EPC);
      if constexpr (WT == 0) {
        *reinterpret_cast<u32x4_t*>(Bs + row * kLDK + kc * 8) = rb[i];
      } else {
        const uint32_t w4[4] = {rb[i].x, rb[i].y, rb[i].z, rb[i].w};
        u32x4_t lo, hi;
        lo.x = e4m3x2_to_bf16x2_m<false>(w4[0]); lo.y = e4m3x2_to_bf16x2_m<true>(w4[0]);
        lo.z = e4m3x2_to_bf16x2_m<false>(w4[1]); lo.w = e4m3x2_to_bf16x2_m<true>(w4[1]);
        hi.x = e4m3x2_to_bf16x2_m<false>(w4[2]); hi.y = e4m3x2_to_bf16x2_m<true>(w4[2]);
        hi.z = e4m3x2_to_bf16x2_m<false>(w4[3]); hi.w = e4m3x2_to_bf16x2_m<true>(w4[3]);
        *reinterpret_cast<u32x4_t*>(Bs + row * kLDK + kc * 16) = lo;
        *reinterpret_cast<u32x4_t*>(Bs + row * kLDK + kc * 16 + 8) = hi;
      }
    }
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  if (K > 0) {
    load(0);
    store();
    __syncthreads();
  }
  for (int k0 = 0; k0 < K; k0 += kBK) {
    const bool next = k0 + kBK < K;
    if (next) load(k0 + kBK);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(
            As + (wm * TM + i * 32 + (lane & 31)) * kLDK + kk * 16 + 8 * (lane >> 5));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(
            Bs + (wn * TN + j * 32 + (lane & 31)) * kLDK + kk * 16 + 8 * (lane >> 5));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
    if (next) {
      store();
      __syncthreads();
    }
  }

  // ---- epilogue -----------------------------------------------------------
  // Row of accumulator r in fragment (i, j): 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lrow = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      const int row = m0 + lrow;
      float rmax = 0.0f;
      unsigned long long rkey = 0ull;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int lcol = wn * TN + j * 32 + (lane & 31);
        const int col = n0 + lcol;
        if (row < M && col < n) {
          const float dot = acc[i][j][r];
          if constexpr (EPI == kEpiCloud) {
            float zv = dot;
            if constexpr (WT == 1) zv = zv * a.wscale[s_ids[lcol]];
            if (a.bias) zv = zv + a.bias[s_ids[lcol]];
            a.z[(int64_t)row * n + col] = zv;
            rmax = fmaxf(rmax, fabsf(fminf(fmaxf(zv, -a.clip), a.clip)));
          } else {
            const float f = __builtin_fmaf((float)a.q[(int64_t)row * n + col], a.qscale[row], dot);
            if (a.f) a.f[(int64_t)row * n + col] = f;
            const unsigned long long key = argmax_key_m(f, col);
            rkey = key > rkey ? key : rkey;
          }
        }
      }
      // fold the 32 lanes that share this row
      if constexpr (EPI == kEpiCloud) {
#pragma unroll
        for (int o = 16; o >= 1; o >>= 1) rmax = fmaxf(rmax, __shfl_xor(rmax, o, 64));
        if ((lane & 31) == 0) atomicMax(&s_rmax[lrow], __float_as_uint(rmax));
      } else {
#pragma unroll
        for (int o = 16; o >= 1; o >>= 1) {
          const unsigned long long y = shfl_xor_u64_m(rkey, o);
          rkey = y > rkey ? y : rkey;
        }
        if ((lane & 31) == 0) atomicMax(&s_rkey[lrow], rkey);
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < BM; i += NT) {
    const int row = m0 + i;
    if (row >= M) continue;
    if constexpr (EPI == kEpiCloud)
      a.amax_part[(int64_t)row * kMaxBlocks + nt] = __uint_as_float(s_rmax[i]);
    else
      a.best_part[(int64_t)row * kMaxBlocks + nt] = s_rkey[i];
  }
}

template <int BM, int BN, int WM, int WN, int WT, int EPI>
static hipError_t launch_tile(MfmaArgs a, hipStream_t s) {
  a.m_tiles = (a.M + BM - 1) / BM;
  a.n_tiles = (a.n + BN - 1) / BN;
  if (a.n_tiles > kMaxBlocks) return hipErrorInvalidValue;
  hipLaunchKernelGGL((k_mfma<BM, BN, WM, WN, WT, EPI>), dim3(a.m_tiles * a.n_tiles),
                     dim3(64 * WM * WN), 0, s, a);
  return hipGetLastError();
}

int mfma_n_tiles(int n) { return (n + kMfmaBN - 1) / kMfmaBN; }

hipError_t launch_mfma(int epi, int wtype, const MfmaArgs& a, hipStream_t s) {
  if (epi == kEpiCloud)
    return wtype == 0 ? launch_tile<128, kMfmaBN, 2, 2, 0, kEpiCloud>(a, s)
                      : launch_tile<128, kMfmaBN, 2, 2, 1, kEpiCloud>(a, s);
  if (wtype != 0) return hipErrorInvalidValue;
  return launch_tile<128, kMfmaBN, 2, 2, 0, kEpiFuse>(a, s);
}

}  // namespace sph
