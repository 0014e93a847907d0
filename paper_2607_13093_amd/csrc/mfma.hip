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
// and the tile's per-row (value, position) argmax key.  The endpoint
// projection with K a multiple of the K step (k_fuse_dma) computes the
// transposed tile, so that a lane holds consecutive subset positions of one
// row: four payload codes per LDS read and an argmax that stays in the lane.
#include <atomic>
#include <type_traits>

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

constexpr int kBK = 64;          // K elements per staged step
constexpr int kLDK = kBK + 8;    // padded LDS row, bf16 elements (144 bytes)
constexpr int kGM = 8;           // m-tiles grouped per n-tile in the tile order

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


// Lane exchanges of the butterfly below, all VALU except the 4-lane step:
// v_permlane16_swap exchanges the upper 16 lanes of each 32-lane half of one
// register with the lower 16 of another, so the larger of its two results is,
// in lanes l & 16 == 0, max(x[l], x[l ^ 16]) and otherwise max(y[l], y[l ^ 16]);
// DPP row_ror:8 and quad permutations read lane l ^ 8, l ^ 2 and l ^ 1.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int O>
__device__ __forceinline__ uint32_t lane_xor_u32(uint32_t v) {
  if constexpr (O == 8) return dpp_u32<0x128>(v);       // row_ror:8
  else if constexpr (O == 2) return dpp_u32<0x4E>(v);   // quad_perm 2,3,0,1
  else if constexpr (O == 1) return dpp_u32<0xB1>(v);   // quad_perm 1,0,3,2
  else return (uint32_t)__shfl_xor((int)v, O, 64);
}
template <class T>
__device__ __forceinline__ T vmax(T a, T b) { return a > b ? a : b; }

// The 64-bit value of lane l ^ 32.
// v of lane l ^ 32: a permlane32 swap trades lanes [32, 64) of its first
// operand with lanes [0, 32) of its second, so with v in both a low lane
// finds its partner's value in the second result, a high lane in the first
__device__ __forceinline__ unsigned long long xor_lane_u64_32(unsigned long long v) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  const auto sl = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
  const auto sh = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  const bool low = (threadIdx.x & 32) == 0;
  return ((unsigned long long)(low ? sh[1] : sh[0]) << 32) | (low ? sl[1] : sl[0]);
}

// Values are float or 64-bit keys, moved as 32-bit words.
template <class T, int O>
__device__ __forceinline__ T xor_lane(T v) {
  if constexpr (sizeof(T) == 8) {
    const uint32_t lo = lane_xor_u32<O>((uint32_t)v), hi = lane_xor_u32<O>((uint32_t)(v >> 32));
    return ((T)hi << 32) | lo;
  } else {
    return __uint_as_float(lane_xor_u32<O>(__float_as_uint(v)));
  }
}
template <class T>
__device__ __forceinline__ void swap16(T& x, T& y) {
  if constexpr (sizeof(T) == 8) {
    const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)x, (uint32_t)y, false, false);
    const auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(x >> 32), (uint32_t)(y >> 32), false, false);
    x = ((T)hi[0] << 32) | lo[0];
    y = ((T)hi[1] << 32) | lo[1];
  } else {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    x = __uint_as_float(r[0]);
    y = __uint_as_float(r[1]);
  }
}

template <int O, int CNT, int P, class T>
__device__ __forceinline__ void half_wave_max_step(T (&v)[P], int lane) {
  if constexpr (O >= 1) {
    constexpr int H = CNT / 2;
    const bool upper = (lane & O) != 0;
#pragma unroll
    for (int i = 0; i < H; ++i) {
      if constexpr (O == 16) {
        T x = v[i], y = v[i + H];
        swap16(x, y);
        v[i] = vmax(x, y);
      } else {
        const T t0 = vmax(v[i], xor_lane<T, O>(v[i]));
        const T t1 = vmax(v[i + H], xor_lane<T, O>(v[i + H]));
        v[i] = upper ? t1 : t0;
      }
    }
    half_wave_max_step<O / 2, H, P>(v, lane);
  }
}

// Transposing butterfly inside each 32-lane half of a wave: on entry lane l
// holds P values; after log2(32) exchanges lane (l & 31) holds the max over
// the half's 32 lanes of values (l & 31) * P/32 .. + P/32 - 1.
template <int P, class T>
__device__ __forceinline__ void half_wave_max_transpose(T (&v)[P], int lane) {
  static_assert(P >= 32 && P % 32 == 0, "values per lane");
  half_wave_max_step<16, P, P>(v, lane);
}

// Epilogue of a BM x BN tile held as acc[FM][FN] 32x32 fragments by the
// WM x WN waves.  Row of accumulator r in fragment (i, j):
// 8*(r/4) + 4*(lane/32) + r%4; column: lane % 32.
// For the fuse epilogue the payload tile q[m0:m0+BM, n0:n0+BN] and the row
// scales are first staged in LDS the main loop no longer needs (s_q: BM*BN
// bytes, s_qs: BM payload scales, then BM factors of the dot products: the
// hidden-state code scales, or 1) with coalesced loads, instead of one byte load per
// accumulator.  The caller has passed a barrier after its last LDS read.
// z of one accumulator: fp8 row scale, then the bias (eq. 12)
// A pointer that is the same in every lane, made visibly uniform (scalar
// registers) so that memory instructions can take it as their scalar base.
__device__ __forceinline__ const uint8_t* scalar_ptr(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t*>(((uint64_t)hi << 32) | lo);
}

template <int WT>
__device__ __forceinline__ float cloud_value(float dot, const MfmaArgs& a, int id) {
  float zv = dot;
  if constexpr (WT == 1) zv = zv * a.wscale[id];
  if (a.bias) zv = zv + a.bias[id];
  return zv;
}

template <int BM, int BN, int WM, int WN, int WT, int EPI, int FM, int FN>
__device__ __forceinline__ void tile_epilogue(f32x16_t (&acc)[FM][FN], const MfmaArgs& a,
                                              const int32_t* s_ids, uint32_t* s_rmax,
                                              unsigned long long* s_rkey, int m0, int n0,
                                              int nt, int8_t* s_q, float* s_qs) {
  constexpr int NT = 64 * WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int P = (FM * 16 + 31) / 32 * 32;  // row values per lane, padded for the butterfly
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = a.M, n = a.n;
  if constexpr (EPI == kEpiFuse) {
    // the payload tile: BN codes of a row are BN * qbits / 8 bytes starting
    // at byte n0 * qbits / 8 of the row
    const int qb = a.qbits;
    const int TB = BN * qb / 8;  // tile bytes per row
    const int64_t c0 = (int64_t)n0 * qb / 8;
    const int64_t rowbytes = ((int64_t)n * qb + 7) / 8;
    const bool vec = (a.qstride & 15) == 0 && (reinterpret_cast<uintptr_t>(a.q) & 15) == 0;
    if (vec) {
      // all of a thread's 16-byte chunks are loaded before any is stored
      constexpr int PT = BM * (BN / 16) / NT;  // chunks per thread at 8 bits
      static_assert(PT * NT == BM * (BN / 16), "payload tile / threads");
      const int CPR = TB / 16;  // 16-byte chunks per tile row
      u32x4_t v[PT];
#pragma unroll
      for (int t = 0; t < PT; ++t) {
        const int c = tid + t * NT, r = c / CPR, k = c % CPR;
        const int row = m0 + r;
        const int64_t col = c0 + k * 16;
        v[t] = (r < BM && row < M && col < rowbytes)
                   ? *reinterpret_cast<const u32x4_t*>(a.q + (int64_t)row * a.qstride + col)
                   : u32x4_t{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int t = 0; t < PT; ++t) {
        const int c = tid + t * NT, r = c / CPR, k = c % CPR;
        if (r < BM) *reinterpret_cast<u32x4_t*>(s_q + r * TB + k * 16) = v[t];
      }
    } else {
      for (int c = tid; c < BM * TB; c += NT) {
        const int r = c / TB, k = c % TB;
        const int row = m0 + r;
        const int64_t col = c0 + k;
        s_q[c] = (row < M && col < rowbytes) ? (int8_t)a.q[(int64_t)row * a.qstride + col] : (int8_t)0;
      }
    }
    // a tile lies in one block of positions (blocks are multiples of BN)
    const int kb = a.qshift < 0 ? 0 : (n0 >> a.qshift);
    for (int r = tid; r < BM; r += NT) {
      s_qs[r] = m0 + r < M ? a.qscale[(int64_t)(m0 + r) * a.qnb + kb] : 0.0f;
      s_qs[BM + r] = (a.hscale && m0 + r < M) ? a.hscale[m0 + r] : 1.0f;
    }
    __syncthreads();
  }
  constexpr bool kCloud = EPI != kEpiFuse;  // kEpiCloud or kEpiCloudQ
  using V = typename std::conditional<kCloud, float, unsigned long long>::type;
  V red[P];
#pragma unroll
  for (int t = FM * 16; t < P; ++t) red[t] = V(0);
  auto fill = [&]() {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lrow = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int row = m0 + lrow;
        V best = V(0);
        // fuse: the lane's largest fused value of the row and its column (the
        // first, so the lowest, of equal values); one key per row afterwards
        float bv = 0.0f;
        int bc = -1;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int lcol = wn * TN + j * 32 + (lane & 31);
          const int col = n0 + lcol;
          if (row < M && col < n) {
            const float dot = acc[i][j][r];
            if constexpr (kCloud) {
              const float zv = cloud_value<WT>(dot, a, s_ids[lcol]);
              if (EPI == kEpiCloud || a.z) __builtin_nontemporal_store(zv, a.z + (int64_t)row * n + col);
              best = fmaxf(best, fabsf(fminf(fmaxf(zv, -a.clip), a.clip)));
            } else {
              int code;
              if (a.qbits == 8) {
                code = s_q[lrow * BN + lcol];
              } else {
                const int byte = (uint8_t)s_q[lrow * (BN / 2) + (lcol >> 1)];
                const int nib = (lcol & 1) ? (byte >> 4) : (byte & 15);
                code = nib >= 8 ? nib - 16 : nib;
              }
              const float f = __builtin_fmaf((float)code, s_qs[lrow], dot * s_qs[BM + lrow]);
              if (a.f) __builtin_nontemporal_store(f, a.f + (int64_t)row * n + col);
              if (bc < 0 || f > bv) {
                bv = f;
                bc = col;
              }
            }
          }
        }
        if constexpr (!kCloud) best = bc >= 0 ? argmax_key_m(bv, bc) : 0ull;
        red[i * 16 + r] = best;
      }
    }
  };
  // Cloud tiles wholly inside z: the same values and row maxima without a
  // bounds test per element.  Each store is the scalar-base + 32-bit-offset
  // form (the row's base is uniform, the lane adds its column and, for lanes
  // 32..63, the four rows below), and max |clamp(z)| is taken as
  // min(|z|, c), which is the same value for every z, NaN included.  The
  // general form above compiled to two branches, a 64-bit address and a
  // reload of the bias pointer per element: 13.6 us of a 210 us block on
  // the dense 2048-row shape.
  auto fill_full = [&](auto has_bias, auto store) {
    constexpr bool HB = decltype(has_bias)::value, ST = decltype(store)::value;
    float cs[FN], cb[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int id = s_ids[wn * TN + j * 32 + (lane & 31)];
      cs[j] = WT == 1 ? a.wscale[id] : 1.0f;
      cb[j] = HB ? a.bias[id] : 0.0f;
    }
    uint32_t loff = ((uint32_t)(lane >> 5) * 4u * (uint32_t)n + (uint32_t)(lane & 31)) * 4u;
    asm volatile("" : "+v"(loff));
    const float clip = a.clip;
    const int row0 = __builtin_amdgcn_readfirstlane(m0 + wm * TM);  // first row of the wave's tile
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + i * 32 + 8 * (r >> 2) + (r & 3);  // the row of lanes 0..31
        const uint8_t* rb = scalar_ptr(a.z + (int64_t)row * n + n0 + wn * TN);
        float best = 0.0f;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          float zv = acc[i][j][r];
          if constexpr (WT == 1) zv = zv * cs[j];
          if constexpr (HB) zv = zv + cb[j];
          if constexpr (ST)
            __builtin_nontemporal_store(zv, (__attribute__((address_space(1))) float*)(rb + loff + j * 128));
          best = fmaxf(best, fminf(fabsf(zv), clip));
        }
        red[i * 16 + r] = V(best);
      }
    }
  };
  bool done = false;
  if constexpr (kCloud) {
    if (m0 + BM <= M && n0 + BN <= n && n <= (1 << 27)) {
      const bool st = EPI == kEpiCloud || a.z != nullptr;
      if (a.bias) {
        if (st) fill_full(std::true_type{}, std::true_type{});
        else fill_full(std::true_type{}, std::false_type{});
      } else {
        if (st) fill_full(std::false_type{}, std::true_type{});
        else fill_full(std::false_type{}, std::false_type{});
      }
      done = true;
    }
  }
  if (!done) fill();
  half_wave_max_transpose<P>(red, lane);
  constexpr int PER = P / 32;
#pragma unroll
  for (int t = 0; t < PER; ++t) {
    const int idx = (lane & 31) * PER + t;
    if (idx >= FM * 16) continue;
    const int i = idx / 16, r = idx % 16;
    const int lrow = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    if constexpr (kCloud)
      atomicMax(&s_rmax[lrow], __float_as_uint(red[t]));
    else
      atomicMax(&s_rkey[lrow], red[t]);
  }
  __syncthreads();
  if constexpr (EPI == kEpiCloudQ) {
    // The tile is one scale block of every row: s = a / qmax from the tile's
    // row maximum of |clamp(z)|, codes rint(clamp(z) / s) from the
    // accumulators still in registers (the same fp32 operations as the
    // quantiser kernel), one byte per code in LDS (the A staging area), then
    // stored row by row, two codes per byte for b = 4; codes of positions
    // past n are 0 (the pad nibble).
    const float qmax = a.qout_bits == 8 ? 127.0f : 7.0f;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lrow = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const float sc = __uint_as_float(s_rmax[lrow]) / qmax;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int lcol = wn * TN + j * 32 + (lane & 31);
          int code = 0;
          if (n0 + lcol < n) {
            const float y = fminf(fmaxf(cloud_value<WT>(acc[i][j][r], a, s_ids[lcol]), -a.clip), a.clip);
            const float t = sc > 0.0f ? y / sc : 0.0f;
            code = (int)fminf(fmaxf(rintf(t), -qmax), qmax);
          }
          s_q[lrow * BN + lcol] = (int8_t)code;
        }
      }
    }
    __syncthreads();
    const int bits = a.qout_bits;
    const int TB = BN * bits / 8;                      // code bytes of a tile row
    const int64_t c0 = (int64_t)n0 * bits / 8;
    const int64_t rowbytes = ((int64_t)n * bits + 7) / 8;
    const bool vec = (a.qout_stride & 15) == 0 && (reinterpret_cast<uintptr_t>(a.qout) & 15) == 0;
    for (int c = tid; c < BM * (TB / 16); c += NT) {
      const int r = c / (TB / 16), k = c % (TB / 16);
      const int row = m0 + r;
      const int64_t col = c0 + (int64_t)k * 16;
      if (row >= M || col >= rowbytes) continue;
      uint32_t wv[4];
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        uint32_t w = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int byte = 4 * e4 + e;
          uint32_t v;
          if (bits == 8) {
            v = (uint8_t)s_q[r * BN + k * 16 + byte];
          } else {
            const int p0 = k * 32 + 2 * byte;
            v = ((uint32_t)s_q[r * BN + p0] & 15u) | (((uint32_t)s_q[r * BN + p0 + 1] & 15u) << 4);
          }
          w |= v << (8 * e);
        }
        wv[e4] = w;
      }
      uint8_t* dst = a.qout + (int64_t)row * a.qout_stride + col;
      if (vec && col + 16 <= rowbytes) {
        *reinterpret_cast<u32x4_t*>(dst) = u32x4_t{wv[0], wv[1], wv[2], wv[3]};
      } else {
        for (int b = 0; b < 16 && col + b < rowbytes; ++b) dst[b] = (uint8_t)(wv[b >> 2] >> (8 * (b & 3)));
      }
    }
    for (int i = tid; i < BM; i += NT) {
      const int row = m0 + i;
      if (row < M) a.qout_scale[(int64_t)row * a.qout_nb + nt] = __uint_as_float(s_rmax[i]) / qmax;
    }
    return;
  }
  for (int i = tid; i < BM; i += NT) {
    const int row = m0 + i;
    if (row >= M) continue;
    if constexpr (kCloud)
      a.amax_part[(int64_t)row * kMaxBlocks + nt] = __uint_as_float(s_rmax[i]);
    else
      a.best_part[(int64_t)row * kMaxBlocks + nt] = s_rkey[i];
  }
}

// BM x BN tile per block, 4 waves in a 2 x 2 grid, wave tile (BM/2) x (BN/2).
// LDS holds two K steps of both tiles; the global loads of step k+1 are in
// flight (in registers) while step k's MFMAs run, then land in the other LDS
// buffer, so each step needs a single barrier.
template <int BM, int BN, int WT, int EPI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_mfma(const MfmaArgs a) {
  constexpr int NT = 256;
  constexpr int TM = BM / 2, TN = BN / 2;    // wave tile
  constexpr int FM = TM / 32, FN = TN / 32;  // 32x32 fragments per wave
  constexpr int A_CH = BM * (kBK / 8) / NT;  // 16-byte A chunks per thread per step
  constexpr int B_EPC = WT == 0 ? 8 : 16;    // weight elements per 16-byte chunk
  constexpr int B_CH = BN * (kBK / B_EPC) / NT;
  static_assert(A_CH * NT == BM * (kBK / 8) && B_CH * NT == BN * (kBK / B_EPC), "tile/threads");

  extern __shared__ __align__(16) uint8_t smem[];
  uint16_t* As = reinterpret_cast<uint16_t*>(smem);            // [2][BM][kLDK]
  uint16_t* Bs = As + 2 * BM * kLDK;                             // [2][BN][kLDK]
  int32_t* s_ids = reinterpret_cast<int32_t*>(Bs + 2 * BN * kLDK);
  uint32_t* s_rmax = reinterpret_cast<uint32_t*>(s_ids + BN);
  unsigned long long* s_rkey = reinterpret_cast<unsigned long long*>(s_rmax + BM + (BM & 1));

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
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
  auto store = [&](int buf) {
    uint16_t* as = As + buf * BM * kLDK;
    uint16_t* bs = Bs + buf * BN * kLDK;
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + i * NT, row = c >> 3, kc = c & 7;
      *reinterpret_cast<u32x4_t*>(as + row * kLDK + kc * 8) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + i * NT;
      const int row = c / (kBK / B_EPC), kc = c % (kBK / B_EPC);
      if constexpr (WT == 0) {
        *reinterpret_cast<u32x4_t*>(bs + row * kLDK + kc * 8) = rb[i];
      } else {
        const uint32_t w4[4] = {rb[i].x, rb[i].y, rb[i].z, rb[i].w};
        u32x4_t lo, hi;
        lo.x = e4m3x2_to_bf16x2_m<false>(w4[0]); lo.y = e4m3x2_to_bf16x2_m<true>(w4[0]);
        lo.z = e4m3x2_to_bf16x2_m<false>(w4[1]); lo.w = e4m3x2_to_bf16x2_m<true>(w4[1]);
        hi.x = e4m3x2_to_bf16x2_m<false>(w4[2]); hi.y = e4m3x2_to_bf16x2_m<true>(w4[2]);
        hi.z = e4m3x2_to_bf16x2_m<false>(w4[3]); hi.w = e4m3x2_to_bf16x2_m<true>(w4[3]);
        *reinterpret_cast<u32x4_t*>(bs + row * kLDK + kc * 16) = lo;
        *reinterpret_cast<u32x4_t*>(bs + row * kLDK + kc * 16 + 8) = hi;
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
    store(0);
    __syncthreads();
  }
  int buf = 0;
  for (int k0 = 0; k0 < K; k0 += kBK) {
    const bool next = k0 + kBK < K;
    if (next) load(k0 + kBK);
    const uint16_t* as = As + buf * BM * kLDK;
    const uint16_t* bs = Bs + buf * BN * kLDK;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(
            as + (wm * TM + i * 32 + (lane & 31)) * kLDK + kk * 16 + 8 * (lane >> 5));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(
            bs + (wn * TN + j * 32 + (lane & 31)) * kLDK + kk * 16 + 8 * (lane >> 5));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    // The other buffer was last read in the previous step, which every wave
    // finished before the barrier that ended it.
    if (next) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  tile_epilogue<BM, BN, 2, 2, WT, EPI>(acc, a, s_ids, s_rmax, s_rkey, m0, n0, nt,
                                 reinterpret_cast<int8_t*>(As), reinterpret_cast<float*>(Bs));
}


// Direct-to-LDS variant (bf16 weights, K a multiple of 64).  gfx950's
// global_load_lds_dwordx4 writes a wave's 64 x 16 bytes straight into LDS
// (lane l at base + 16*l), so tiles never pass through registers and no
// ds_write is issued.  A wave instruction fills 8 rows x 128 bytes; rows are
// unpadded and their 16-byte chunks are XOR-swizzled with
// f(row) = (row & 7) ^ ((row >> 3) & 1), which keeps every fragment read
// conflict-free whether the LDS serves 8 or 16 lanes per cycle.  Rows past
// M and subset positions past n read a valid row (row M-1 / the last id):
// they only feed outputs that are never written.  On the decode-sized dense
// shape this loop ran 1.2x faster than register staging.
// Waves: WM x WN (wave tile (BM/WM) x (BN/WN)); 2 x 2 with one wave per SIMD,
// or 2 x 4 for 320-row tiles (wave tile 160 x 64) with two waves per SIMD,
// whose accumulators then live in the 256 registers each wave has.
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ int swz8(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// Copy addressing of the direct-to-LDS kernels.  With O32 every lane keeps
// its row's byte offset (below 4 GiB) in a 32-bit register and the step's
// base stays scalar: each copy is then the scalar-base + 32-bit-offset form
// of global_load_lds with no address arithmetic of its own (the empty asm
// keeps the compiler from folding the base into 64-bit lane addresses, which
// costs a 64-bit add per copy and chains the copies through one register
// pair).  Measured on dense_sub's cloud projection: 1106 -> 1033 us.

template <bool O32>
struct LaneAddr;
template <>
struct LaneAddr<true> {
  uint32_t off;
  __device__ __forceinline__ void set(const uint8_t*, int64_t o) { off = (uint32_t)o; }
  // base: the step's scalar base (from scalar_ptr)
  __device__ __forceinline__ void copy(const uint8_t* base, int64_t, lds_void_t* dst) {
    asm volatile("" : "+v"(off));
    __builtin_amdgcn_global_load_lds(base + off, dst, 16, 0, 0);
  }
};
template <>
struct LaneAddr<false> {
  const uint8_t* p;
  __device__ __forceinline__ void set(const uint8_t* base, int64_t o) { p = base + o; }
  __device__ __forceinline__ void copy(const uint8_t*, int64_t step, lds_void_t* dst) {
    __builtin_amdgcn_global_load_lds(p + step, dst, 16, 0, 0);
  }
};

template <int BM, int BN, int WM, int WN, int EPI, bool O32>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(WM * WN / 4, WM * WN / 4)))
void k_mfma_dma(const MfmaArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int NT = 64 * WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  // With two waves per SIMD only the first wave of each SIMD issues the
  // copies (all of them): a copy instruction can hold its wave at issue
  // until the load path accepts it, and the SIMD's other wave keeps the
  // matrix pipe busy meanwhile.  Measured on the dense 2048-row shape: 3-5%
  // faster than all 8 waves issuing an eighth of the copies each.
  constexpr int IW = WM * WN >= 8 ? WM * WN / 2 : WM * WN;
  constexpr int A_INS = BM / 8 / IW, B_INS = BN / 8 / IW;  // copy instructions per issuing wave per step
  static_assert(A_INS * 8 * IW == BM && B_INS * 8 * IW == BN, "tile rows / issuing waves");
  extern __shared__ __align__(16) uint8_t smem[];
  uint16_t* As = reinterpret_cast<uint16_t*>(smem);      // [2][BM][64]
  uint16_t* Bs = As + 2 * BM * kBK;                       // [2][BN][64]
  int32_t* s_ids = reinterpret_cast<int32_t*>(Bs + 2 * BN * kBK);
  uint32_t* s_rmax = reinterpret_cast<uint32_t*>(s_ids + BN);
  unsigned long long* s_rkey = reinterpret_cast<unsigned long long*>(s_rmax + BM + (BM & 1));

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int iw = wave < IW ? wave : 0;  // issuing slot (waves >= IW issue nothing)
  const int wm = wave / WN, wn = wave % WN;
  int mt, nt;
  tile_of_block(blockIdx.x, a.m_tiles, a.n_tiles, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int M = a.M, K = a.K, n = a.n;
  const int last_id = a.ids[min(n, n0 + BN) - 1];
  for (int i = tid; i < BN; i += NT) s_ids[i] = n0 + i < n ? a.ids[n0 + i] : last_id;
  for (int i = tid; i < BM; i += NT) {
    s_rmax[i] = 0u;
    s_rkey[i] = 0ull;
  }
  __syncthreads();

  // lane -> row (lane / 8) of its 8-row group and the logical chunk it fetches
  const int lr = lane >> 3;
  const uint8_t* hbase = reinterpret_cast<const uint8_t*>(a.h);
  LaneAddr<O32> pa[A_INS], pb[B_INS];
#pragma unroll
  for (int i = 0; i < A_INS; ++i) {
    const int r = (iw * A_INS + i) * 8 + lr;
    const int lc = (lane & 7) ^ swz8(r);
    pa[i].set(hbase, (int64_t)min(m0 + r, M - 1) * a.ldh * 2 + lc * 16);
  }
#pragma unroll
  for (int i = 0; i < B_INS; ++i) {
    const int r = (iw * B_INS + i) * 8 + lr;
    const int lc = (lane & 7) ^ swz8(r);
    pb[i].set(a.w, (int64_t)s_ids[r] * a.ldw_bytes + lc * 16);
  }
  auto issue = [&](int k0, int stage) {
    if (wave >= IW) return;
    uint8_t* as = reinterpret_cast<uint8_t*>(As + stage * BM * kBK);
    uint8_t* bs = reinterpret_cast<uint8_t*>(Bs + stage * BN * kBK);
    const int64_t step = (int64_t)k0 * 2;
    const uint8_t* ha = O32 ? scalar_ptr(hbase + step) : nullptr;
    const uint8_t* wb = O32 ? scalar_ptr(a.w + step) : nullptr;
#pragma unroll
    for (int i = 0; i < A_INS; ++i) pa[i].copy(ha, step, (lds_void_t*)(as + (iw * A_INS + i) * 1024));
#pragma unroll
    for (int i = 0; i < B_INS; ++i) pb[i].copy(wb, step, (lds_void_t*)(bs + (iw * B_INS + i) * 1024));
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  if (K > 0) {
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  int stage = 0;
  for (int k0 = 0; k0 < K; k0 += kBK) {
    // the other stage was last read in the previous step, finished by all
    // waves before that step's closing barrier
    if (k0 + kBK < K) issue(k0 + kBK, stage ^ 1);
    const uint16_t* as = As + stage * BM * kBK;
    const uint16_t* bs = Bs + stage * BN * kBK;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8_t af[FM], bfr[FN];
      const int c = kk * 2 + (lane >> 5);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * TM + i * 32 + (lane & 31);
        af[i] = *reinterpret_cast<const bf16x8_t*>(as + row * kBK + ((c ^ swz8(row)) << 3));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int row = wn * TN + j * 32 + (lane & 31);
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(bs + row * kBK + ((c ^ swz8(row)) << 3));
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's loads for the next stage have landed
    __syncthreads();
    stage ^= 1;
  }
  tile_epilogue<BM, BN, WM, WN, 0, EPI>(acc, a, s_ids, s_rmax, s_rkey, m0, n0, nt,
                                reinterpret_cast<int8_t*>(As), reinterpret_cast<float*>(Bs));
#endif
}

// One wave per SIMD for the dense bf16 cloud projection (256 x 256 tiles, an
// even number, at least 2, of 64-wide K steps).  Four waves, each a 128 x 128 wave tile of
// 4 x 4 fragments whose 256 accumulators stay in the AGPRs: per 16-wide
// sub-step a wave reads 8 fragments for 16 MFMAs, where the two-wave kernel
// reads 6 for 8, so the LDS traffic per flop drops by a third.  With no second
// wave on the SIMD the schedule is explicit: the MFMAs and the LDS fragment
// reads are inline asm (their order is kept as written).  Four fragment
// register sets, one per sub-step: while a sub-step's 16 MFMAs issue, the
// reads for the sub-step two ahead go out after its first 8 MFMAs, into the
// set the MFMAs of two sub-steps ago used.  One barrier per step, between the
// second and third sub-steps: the third and fourth then read the next stage
// and (two weight stages) copy the step after next into this one, 8 copies
// each; three weight stages spread the copies differently (below).  Past the end
// the copies repeat the last step (in-bounds reads into a stage nobody reads),
// so the K loop is straight-line code: with a branch in it the compiler
// spilled registers that reads still in flight were to fill.  The compiler
// sees neither the asm reads nor the MFMAs, so every wait is explicit
// (lgkmcnt before each sub-step's MFMAs, vmcnt and lgkmcnt before the
// barrier), and each sub-step's fragments stay allocated to its end.
// Measured (harness, dense_full / dense_sub): reads one sub-step ahead with
// two sets 3397 / 1022 us, two ahead with four sets 3300 / 970 us.
__device__ __forceinline__ void w1_mfma(f32x16_t& c, const bf16x8_t& a, const bf16x8_t& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}
template <int OFF>
__device__ __forceinline__ void w1_read(bf16x8_t& d, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(d) : "v"(addr), "i"(OFF));
}
__device__ __forceinline__ void w1_wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// the older of two groups of 8 reads (LDS reads complete in order)
__device__ __forceinline__ void w1_wait_lds8() { asm volatile("s_waitcnt lgkmcnt(8)" ::: "memory"); }
__device__ __forceinline__ void w1_wait_mem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
typedef __attribute__((address_space(3))) const char* lds_cptr_t;


// NB weight stages: 2 (an even number of K steps; 128 KB of LDS), or 3 (a
// multiple of 6 steps; all 160 KB of LDS, and the ids and row maxima live
// outside the stages: ids are read from global memory, the row maxima take
// the first stage after the K loop).  With three, a step's first two
// sub-steps copy the weights of two steps ahead into the stage the previous
// step read and its last two copy h, one copy per 4 MFMAs in every sub-step,
// so the barrier waits for all but the newest 8 copies (those weights).
// Harness, dense_full / dense_sub: two stages 3300 / 996 us; three, weights
// copied in the last sub-step three steps ahead, 3250 / 970 us; three with
// the copies spread over the step 3290 -> 3257 / 1004 -> 961 us (A/B runs).
template <int EPI, int NB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_mfma_w1(const MfmaArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  static_assert(EPI == kEpiCloud, "cloud epilogue only");
  static_assert(NB == 2 || NB == 3, "two or three weight stages");
  constexpr int BM = 256, BN = 256, NT = 256, WN = 2, TM = 128, TN = 128, FM = 4, FN = 4;
  constexpr int A_INS = BM / 8 / 4, B_INS = BN / 8 / 4;  // 8 + 8 copies per wave per step
  constexpr int SB = BN * kBK * 2;                        // bytes of a stage (32 KB)
  extern __shared__ __align__(16) uint8_t smem[];
  uint8_t* As = smem;                                     // [2][256][128 B]
  uint8_t* Bs = smem + 2 * SB;                            // [NB][256][128 B]
  // ids and row maxima: after the stages (NB = 2), or none / the first stage
  // once the K loop is done (NB = 3)
  int32_t* s_ids = reinterpret_cast<int32_t*>(Bs + NB * SB);
  uint32_t* s_rmax = NB == 2 ? reinterpret_cast<uint32_t*>(s_ids + BN) : reinterpret_cast<uint32_t*>(smem);
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  int mt, nt;
  tile_of_block(blockIdx.x, a.m_tiles, a.n_tiles, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int M = a.M, K = a.K, n = a.n;
  const int S = K / kBK;  // a multiple of 2 (NB = 2) or 6 (NB = 3): the launcher's condition
  const int last_id = a.ids[min(n, n0 + BN) - 1];
  if constexpr (NB == 2) {
    for (int i = tid; i < BN; i += NT) s_ids[i] = n0 + i < n ? a.ids[n0 + i] : last_id;
    for (int i = tid; i < BM; i += NT) s_rmax[i] = 0u;
    __syncthreads();
  }

  const int lr = lane >> 3;
  const uint8_t* hbase = reinterpret_cast<const uint8_t*>(a.h);
  LaneAddr<true> pa[A_INS], pb[B_INS];
#pragma unroll
  for (int i = 0; i < A_INS; ++i) {
    const int r = (wave * A_INS + i) * 8 + lr;
    const int lc = (lane & 7) ^ swz8(r);
    pa[i].set(hbase, (int64_t)min(m0 + r, M - 1) * a.ldh * 2 + lc * 16);
  }
#pragma unroll
  for (int i = 0; i < B_INS; ++i) {
    const int r = (wave * B_INS + i) * 8 + lr;
    const int lc = (lane & 7) ^ swz8(r);
    const int id = NB == 2 ? s_ids[r] : (n0 + r < n ? a.ids[n0 + r] : last_id);
    pb[i].set(a.w, (int64_t)id * a.ldw_bytes + lc * 16);
  }
  // copy i (0..7) of this wave's share of step s into stage st
  auto copyA = [&](int i, int s, int st) {
    const int64_t step = (int64_t)s * kBK * 2;
    pa[i].copy(scalar_ptr(hbase + step), step, (lds_void_t*)(As + st * SB + (wave * A_INS + i) * 1024));
  };
  auto copyB = [&](int i, int s, int st) {
    const int64_t step = (int64_t)s * kBK * 2;
    pb[i].copy(scalar_ptr(a.w + step), step, (lds_void_t*)(Bs + st * SB + (wave * B_INS + i) * 1024));
  };
  // fragment reads: row (lane & 31) of a fragment, 16-byte chunk 2 kk + lane / 32
  // (swizzled); the fragments of a wave are 32 rows (4 KB) apart and the
  // stages 32 KB apart, both immediate offsets of the read (the third weight
  // stage, past the 16-bit offset field, has base addresses of its own)
  uint32_t adA[4], adB[4], adB2[4];
  {
    const int sw = swz8(lane & 31);  // rows 32 apart share the swizzle
    const uint32_t baseA = (uint32_t)(uintptr_t)(lds_cptr_t)As + (uint32_t)((wm * TM + (lane & 31)) * 128);
    const uint32_t baseB = (uint32_t)(uintptr_t)(lds_cptr_t)Bs + (uint32_t)((wn * TN + (lane & 31)) * 128);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint32_t c = (uint32_t)(((kk * 2 + (lane >> 5)) ^ sw) << 4);
      adA[kk] = baseA + c;
      adB[kk] = baseB + c;
      adB2[kk] = baseB + 2u * SB + c;
    }
  }
  f32x16_t acc[FM][FN];
  {
    f32x16_t z0;
#pragma unroll
    for (int r = 0; r < 16; ++r) z0[r] = 0.0f;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) asm volatile("; zero accumulators" : "=a"(acc[i][j]) : "0"(z0));
  }
  bf16x8_t f0a[FM], f0b[FN], f1a[FM], f1b[FN], f2a[FM], f2b[FN], f3a[FM], f3b[FN];
  // read q (0..7) of sub-step KK's fragments (A stage SA, weight stage SW) into set B
  auto rd1 = [&](auto kkc, auto sac, auto swc, auto bc, int q) {
    constexpr int KK = decltype(kkc)::value, SA = decltype(sac)::value, SW = decltype(swc)::value;
    constexpr int B = decltype(bc)::value;
    constexpr int OA = SA * SB, OB = SW == 2 ? 0 : SW * SB;
    const uint32_t ab = SW == 2 ? adB2[KK] : adB[KK];
#define SPH_W1_READ(FA, FB)                             \
    switch (q) {                                        \
      case 0: w1_read<OA + 0>(FA[0], adA[KK]); break;     \
      case 1: w1_read<OB + 0>(FB[0], ab); break;          \
      case 2: w1_read<OA + 4096>(FA[1], adA[KK]); break;  \
      case 3: w1_read<OB + 4096>(FB[1], ab); break;       \
      case 4: w1_read<OA + 8192>(FA[2], adA[KK]); break;  \
      case 5: w1_read<OB + 8192>(FB[2], ab); break;       \
      case 6: w1_read<OA + 12288>(FA[3], adA[KK]); break; \
      default: w1_read<OB + 12288>(FB[3], ab); break;     \
    }
    if constexpr (B == 0) { SPH_W1_READ(f0a, f0b) }
    else if constexpr (B == 1) { SPH_W1_READ(f1a, f1b) }
    else if constexpr (B == 2) { SPH_W1_READ(f2a, f2b) }
    else { SPH_W1_READ(f3a, f3b) }
#undef SPH_W1_READ
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  // the 16 MFMAs of set B, hook(t) after MFMA t; the set stays allocated to the end
  auto phase = [&](auto bc, auto hook) {
    constexpr int B = decltype(bc)::value;
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int i = t >> 2, j = t & 3;
      if constexpr (B == 0) w1_mfma(acc[i][j], f0a[i], f0b[j]);
      else if constexpr (B == 1) w1_mfma(acc[i][j], f1a[i], f1b[j]);
      else if constexpr (B == 2) w1_mfma(acc[i][j], f2a[i], f2b[j]);
      else w1_mfma(acc[i][j], f3a[i], f3b[j]);
      hook(t);
    }
    if constexpr (B == 0)
      asm volatile("" :: "v"(f0a[0]), "v"(f0a[1]), "v"(f0a[2]), "v"(f0a[3]), "v"(f0b[0]), "v"(f0b[1]), "v"(f0b[2]), "v"(f0b[3]));
    else if constexpr (B == 1)
      asm volatile("" :: "v"(f1a[0]), "v"(f1a[1]), "v"(f1a[2]), "v"(f1a[3]), "v"(f1b[0]), "v"(f1b[1]), "v"(f1b[2]), "v"(f1b[3]));
    else if constexpr (B == 2)
      asm volatile("" :: "v"(f2a[0]), "v"(f2a[1]), "v"(f2a[2]), "v"(f2a[3]), "v"(f2b[0]), "v"(f2b[1]), "v"(f2b[2]), "v"(f2b[3]));
    else
      asm volatile("" :: "v"(f3a[0]), "v"(f3a[1]), "v"(f3a[2]), "v"(f3a[3]), "v"(f3b[0]), "v"(f3b[1]), "v"(f3b[2]), "v"(f3b[3]));
  };
  // step s, with h stage SA = s % 2 and weight stage SW = s % NB: the weights
  // for step s + NB and h for step s + 2 are copied into this step's stages
  // after the barrier (past the end: the last step again)
  auto step = [&](auto sac, auto swc, int s) {
    constexpr int SA = decltype(sac)::value, SW = decltype(swc)::value;
    using SAc = std::integral_constant<int, SA>;
    using SWc = std::integral_constant<int, SW>;
    using SAn = std::integral_constant<int, SA ^ 1>;
    using SWn = std::integral_constant<int, (SW + 1) % NB>;
    const int sa = min(s + 2, S - 1), sw = min(s + NB, S - 1);
    // three weight stages: this step's first two sub-steps copy the weights
    // of step s + 2 (4 copies each, one per 4 MFMAs) into the stage step
    // s - 1 read
    constexpr int SWp = (SW + 2) % 3;
    w1_wait_lds8();
    phase(I0{}, [&](int t) {
      if (t < 8) rd1(I2{}, SAc{}, SWc{}, I2{}, t);
      if (NB == 3 && s > 0 && (t & 3) == 1) copyB(t >> 2, sa, SWp);
    });
    w1_wait_lds8();
    phase(I1{}, [&](int t) {
      if (t < 8) rd1(I3{}, SAc{}, SWc{}, I3{}, t);
      if (NB == 3 && s > 0 && (t & 3) == 1) copyB(4 + (t >> 2), sa, SWp);
    });
    // this wave's reads of the stages are done, and its copies for the next
    // step have landed (with three weight stages the newest 8, the weights of
    // step s + 2, may still be in flight)
    w1_wait_lds();
    if constexpr (NB == 2) w1_wait_mem();
    else asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    if constexpr (NB == 2) {
      phase(I2{}, [&](int t) {
        if (t < 8) {
          rd1(I0{}, SAn{}, SWn{}, I0{}, t);
          copyA(t, sa, SA);
        }
      });
      w1_wait_lds8();
      phase(I3{}, [&](int t) {
        if (t < 8) {
          rd1(I1{}, SAn{}, SWn{}, I1{}, t);
          copyB(t, sw, SW);
        }
      });
    } else {
      // h of step s + 2 into this step's h stage, 4 copies per sub-step
      phase(I2{}, [&](int t) {
        if (t < 8) rd1(I0{}, SAn{}, SWn{}, I0{}, t);
        if ((t & 3) == 1) copyA(t >> 2, sa, SA);
      });
      w1_wait_lds8();
      phase(I3{}, [&](int t) {
        if (t < 8) rd1(I1{}, SAn{}, SWn{}, I1{}, t);
        if ((t & 3) == 1) copyA(4 + (t >> 2), sa, SA);
      });
    }
  };
  // prologue: h steps 0 and 1, weight steps 0 .. NB - 1; steps 0 land first
#pragma unroll
  for (int i = 0; i < A_INS; ++i) copyA(i, 0, 0);
#pragma unroll
  for (int i = 0; i < B_INS; ++i) copyB(i, 0, 0);
#pragma unroll
  for (int i = 0; i < A_INS; ++i) copyA(i, 1, 1);
#pragma unroll
  for (int i = 0; i < B_INS; ++i) copyB(i, 1, 1);
  if constexpr (NB == 3) {
#pragma unroll
    for (int i = 0; i < B_INS; ++i) copyB(i, 2, 2);
    asm volatile("s_waitcnt vmcnt(24)" ::: "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 8; ++q) rd1(I0{}, I0{}, I0{}, I0{}, q);
#pragma unroll
  for (int q = 0; q < 8; ++q) rd1(I1{}, I0{}, I0{}, I1{}, q);
  if constexpr (NB == 2) {
    for (int s = 0; s < S; s += 2) {
      step(I0{}, I0{}, s);
      step(I1{}, I1{}, s + 1);
    }
  } else {
    for (int s = 0; s < S; s += 6) {
      step(I0{}, I0{}, s);
      step(I1{}, I1{}, s + 1);
      step(I0{}, I2{}, s + 2);
      step(I1{}, I0{}, s + 3);
      step(I0{}, I1{}, s + 4);
      step(I1{}, I2{}, s + 5);
    }
  }
  // the last copies (into stages nobody reads) and reads land before the
  // LDS is given up; the last MFMAs' results are written before the AGPRs
  // are read
  w1_wait_mem();
  w1_wait_lds();
  asm volatile("s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7" ::: "memory");
  if constexpr (NB == 3) {
    __syncthreads();  // every wave is done with the stages: the row maxima take the first
    for (int i = tid; i < BM; i += NT) s_rmax[i] = 0u;
    __syncthreads();
  }

  // Epilogue: each fragment leaves the AGPRs on its own (the generic tile
  // epilogue, which reads all 256 accumulators, spilled); z and the tile's
  // row maxima of |clamp(z)| as there.
  constexpr int P = FM * 16;
  float red[P];
#pragma unroll
  for (int t = 0; t < P; ++t) red[t] = 0.0f;
  const float clip = a.clip;
  if (m0 + BM <= M && n0 + BN <= n && n <= (1 << 27) && !a.bias) {
    uint32_t loff = ((uint32_t)(lane >> 5) * 4u * (uint32_t)n + (uint32_t)(lane & 31)) * 4u;
    asm volatile("" : "+v"(loff));
    const int row0 = __builtin_amdgcn_readfirstlane(m0 + wm * TM);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        f32x16_t v;
        asm volatile("; fragment out of the AGPRs" : "=v"(v) : "0"(acc[i][j]));
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + i * 32 + 8 * (r >> 2) + (r & 3);
          const uint8_t* rb = scalar_ptr(a.z + (int64_t)row * n + n0 + wn * TN);
          __builtin_nontemporal_store(v[r], (__attribute__((address_space(1))) float*)(rb + loff + j * 128));
          red[i * 16 + r] = fmaxf(red[i * 16 + r], fminf(fabsf(v[r]), clip));
        }
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        f32x16_t v;
        asm volatile("; fragment out of the AGPRs" : "=v"(v) : "0"(acc[i][j]));
        const int lcol = wn * TN + j * 32 + (lane & 31);
        const int col = n0 + lcol;
        float cb = 0.0f;
        if (a.bias) cb = a.bias[NB == 2 ? s_ids[lcol] : (col < n ? a.ids[col] : last_id)];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row < M && col < n) {
            const float zv = a.bias ? v[r] + cb : v[r];
            __builtin_nontemporal_store(zv, a.z + (int64_t)row * n + col);
            red[i * 16 + r] = fmaxf(red[i * 16 + r], fabsf(fminf(fmaxf(zv, -clip), clip)));
          }
        }
      }
    }
  }
  half_wave_max_transpose<P>(red, lane);
  constexpr int PER = P / 32;
#pragma unroll
  for (int t = 0; t < PER; ++t) {
    const int idx = (lane & 31) * PER + t;
    const int i = idx / 16, r = idx % 16;
    const int lrow = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    atomicMax(&s_rmax[lrow], __float_as_uint(red[t]));
  }
  __syncthreads();
  for (int i = tid; i < BM; i += NT)
    if (m0 + i < M) a.amax_part[(int64_t)(m0 + i) * kMaxBlocks + nt] = __uint_as_float(s_rmax[i]);
#endif
}

// Direct-to-LDS variant for fp8 E4M3 weights (K a multiple of 64).  The A
// tile is staged as above; the B tile keeps its bytes: a weight row holds 64
// codes per K step (64 bytes, four 16-byte chunks), and a wave instruction
// fills 16 rows.  Chunks are XOR-swizzled with g(row) = (row >> 2) & 3, so
// the 32 rows a fragment read touches spread over the LDS banks.  Each lane
// reads its 8 codes of a fragment (ds_read_b64) and widens them to bf16
// (exact) in registers right before the MFMA; the per-row scale is applied
// in the epilogue.  With one wave per SIMD all fragments of a step are read
// before the next step's loads are issued (the compiler would otherwise make
// the reads wait for those loads), and scheduling barriers keep the loads
// ahead of the MFMAs.  With two waves per SIMD (320-row tiles) those
// fragments would not fit next to the accumulators: the loads go out first,
// each sub-step reads its own fragments, and the SIMD's other wave covers
// the wait.
__device__ __forceinline__ int swz4(int row) { return (row >> 2) & 3; }

template <int BM, int BN, int WM, int WN, int EPI, bool O32>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(WM * WN / 4, WM * WN / 4)))
void k_mfma_dma8(const MfmaArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int NT = 64 * WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  // as in k_mfma_dma: with two waves per SIMD one of them issues the copies
  constexpr int IW = WM * WN >= 8 ? WM * WN / 2 : WM * WN;
  constexpr int A_INS = BM / 8 / IW, B_INS = BN / 16 / IW;  // copy instructions per issuing wave per step
  static_assert(A_INS * 8 * IW == BM && B_INS * 16 * IW == BN, "tile rows / issuing waves");
  extern __shared__ __align__(16) uint8_t smem[];
  uint16_t* As = reinterpret_cast<uint16_t*>(smem);             // [2][BM][64] bf16
  uint8_t* Bs = reinterpret_cast<uint8_t*>(As + 2 * BM * kBK);   // [2][BN][64] fp8
  int32_t* s_ids = reinterpret_cast<int32_t*>(Bs + 2 * BN * kBK);
  uint32_t* s_rmax = reinterpret_cast<uint32_t*>(s_ids + BN);
  unsigned long long* s_rkey = reinterpret_cast<unsigned long long*>(s_rmax + BM + (BM & 1));

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int iw = wave < IW ? wave : 0;  // issuing slot (waves >= IW issue nothing)
  const int wm = wave / WN, wn = wave % WN;
  int mt, nt;
  tile_of_block(blockIdx.x, a.m_tiles, a.n_tiles, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int M = a.M, K = a.K, n = a.n;
  const int last_id = a.ids[min(n, n0 + BN) - 1];
  for (int i = tid; i < BN; i += NT) s_ids[i] = n0 + i < n ? a.ids[n0 + i] : last_id;
  for (int i = tid; i < BM; i += NT) {
    s_rmax[i] = 0u;
    s_rkey[i] = 0ull;
  }
  __syncthreads();

  const uint8_t* hbase = reinterpret_cast<const uint8_t*>(a.h);
  LaneAddr<O32> pa[A_INS], pb[B_INS];
#pragma unroll
  for (int i = 0; i < A_INS; ++i) {
    const int r = (iw * A_INS + i) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ swz8(r);
    pa[i].set(hbase, (int64_t)min(m0 + r, M - 1) * a.ldh * 2 + lc * 16);
  }
#pragma unroll
  for (int i = 0; i < B_INS; ++i) {
    const int r = (iw * B_INS + i) * 16 + (lane >> 2);
    const int lc = (lane & 3) ^ swz4(r);
    pb[i].set(a.w, (int64_t)s_ids[r] * a.ldw_bytes + lc * 16);
  }
  auto issue = [&](int k0, int stage) {
    if (wave >= IW) return;
    uint8_t* as = reinterpret_cast<uint8_t*>(As + stage * BM * kBK);
    uint8_t* bs = Bs + stage * BN * kBK;
    const uint8_t* ha = O32 ? scalar_ptr(hbase + (int64_t)k0 * 2) : nullptr;
    const uint8_t* wb = O32 ? scalar_ptr(a.w + k0) : nullptr;
#pragma unroll
    for (int i = 0; i < A_INS; ++i)
      pa[i].copy(ha, (int64_t)k0 * 2, (lds_void_t*)(as + (iw * A_INS + i) * 1024));
#pragma unroll
    for (int i = 0; i < B_INS; ++i) pb[i].copy(wb, k0, (lds_void_t*)(bs + (iw * B_INS + i) * 1024));
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  if (K > 0) {
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  int stage = 0;
  for (int k0 = 0; k0 < K; k0 += kBK) {
    const uint16_t* as = As + stage * BM * kBK;
    const uint8_t* bs = Bs + stage * BN * kBK;
    if constexpr (WM * WN > 4) {
      // Two waves per SIMD: a step's fragments for all four sub-steps do not
      // fit in registers next to the accumulators, so the next stage's loads
      // go out first and each sub-step reads its own fragments (the other
      // wave of the SIMD covers any wait on the loads).
      // The step's fp8 codes (8 bytes per fragment and sub-step, 16 VGPRs)
      // are read before the next stage's copies go out.  The compiler makes
      // an LDS read behind pending copies wait for them where it cannot
      // tell the two apart, and it did so for these 8-byte reads: placed
      // after the copies, they held the issuing wave of each SIMD until its
      // copies had landed, every step (sample_fp8 cloud 438 against 365 us).
      uint2 qb[kBK / 16][FN];
#pragma unroll
      for (int kk = 0; kk < kBK / 16; ++kk)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int row = wn * TN + j * 32 + (lane & 31);
          qb[kk][j] = *reinterpret_cast<const uint2*>(bs + row * kBK + ((kk ^ swz4(row)) << 4) + 8 * (lane >> 5));
        }
      if (k0 + kBK < K) issue(k0 + kBK, stage ^ 1);
#pragma unroll
      for (int kk = 0; kk < kBK / 16; ++kk) {
        const int c = kk * 2 + (lane >> 5);
        bf16x8_t af[FM], bfr[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          const int row = wm * TM + i * 32 + (lane & 31);
          af[i] = *reinterpret_cast<const bf16x8_t*>(as + row * kBK + ((c ^ swz8(row)) << 3));
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const uint2 q = qb[kk][j];
          u32x4_t w;
          w.x = e4m3x2_to_bf16x2_m<false>(q.x);
          w.y = e4m3x2_to_bf16x2_m<true>(q.x);
          w.z = e4m3x2_to_bf16x2_m<false>(q.y);
          w.w = e4m3x2_to_bf16x2_m<true>(q.y);
          bfr[j] = __builtin_bit_cast(bf16x8_t, w);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      stage ^= 1;
      continue;
    }
    bf16x8_t af[kBK / 16][FM];
    uint2 bq[kBK / 16][FN];
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int c = kk * 2 + (lane >> 5);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * TM + i * 32 + (lane & 31);
        af[kk][i] = *reinterpret_cast<const bf16x8_t*>(as + row * kBK + ((c ^ swz8(row)) << 3));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int row = wn * TN + j * 32 + (lane & 31);
        bq[kk][j] = *reinterpret_cast<const uint2*>(bs + row * kBK + ((kk ^ swz4(row)) << 4) +
                                                    8 * (lane >> 5));
      }
    }
    // the other stage was last read in the previous step, finished by all
    // waves before that step's closing barrier
    if (k0 + kBK < K) issue(k0 + kBK, stage ^ 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8_t bfr[FN];
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        u32x4_t w;
        w.x = e4m3x2_to_bf16x2_m<false>(bq[kk][j].x);
        w.y = e4m3x2_to_bf16x2_m<true>(bq[kk][j].x);
        w.z = e4m3x2_to_bf16x2_m<false>(bq[kk][j].y);
        w.w = e4m3x2_to_bf16x2_m<true>(bq[kk][j].y);
        bfr[j] = __builtin_bit_cast(bf16x8_t, w);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[kk][i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's loads for the next stage have landed
    __syncthreads();
    stage ^= 1;
  }
  tile_epilogue<BM, BN, WM, WN, 1, EPI>(acc, a, s_ids, s_rmax, s_rkey, m0, n0, nt,
                                reinterpret_cast<int8_t*>(As), reinterpret_cast<float*>(Bs));
#endif
}

// Endpoint projection with its fuse epilogue (eqs. 11, 13-14), K a multiple
// of the K step.  The block computes the transposed tile C^T[n][m] =
// W[S_n] . h[m]: the weight rows are the MFMA's A operand and the rows of h
// its B operand.  The weight rows of each 32-row group are staged in the
// order that puts subset position 16*(l/32) + r of the group in accumulator
// r of lane l: a lane holds 16 consecutive positions of row j*32 + l%32 (in
// the wave's tile) per fragment.  Operands are otherwise staged exactly as
// in k_mfma_dma.  A BM x 256 tile runs WNN x WMM waves (WNN along the
// positions, WMM along the rows).
//
// Payload: the tile's codes (BM rows of 256 * qbits / 8 bytes) are staged
// in LDS as 16-byte chunks, swizzled per row, so one 16-byte read gives a
// lane its 16 8-bit codes (an 8-byte read its 16 4-bit codes) and the rows
// a read touches spread over the banks.  With 8-bit codes on 16-byte
// aligned rows the tile is copied global-to-LDS during the last K step into
// the operand buffers that step does not read (rows [0, BM/2) into the idle
// A buffer, the rest into the idle B buffer), where it lands while the last
// MFMAs run; otherwise it is loaded after the main loop.
//
// Selection: f = fma(code, s, dot * hs) (the product only with hidden-state
// scales), the lane's largest f, then the lowest of the lane's positions
// holding it; the two lanes holding a row (l, l ^ 32) keep the larger
// orderable key (value, then lowest position), and LDS atomics combine the
// WNN waves sharing the row.  Against the row-major epilogue (one LDS byte
// read per code and a 32-lane butterfly of 64-bit keys) the first form of
// this kernel (four positions per register group, a 32-bit code read and a
// running compare per value) ran dense_full's endpoint projection in 358 us
// instead of 505, dense_sub in 85 instead of 114 and batched in 29 instead
// of 47; the 16-position layout then took dense_sub to 81 us and batched to
// 27, with identical keys throughout.  One wave per SIMD instead (the cloud
// kernel's explicit schedule with 128 x 128 wave tiles, the payload copied in
// place of the copies past the end) kept the keys identical but ran slower:
// with 8 K steps a tile's prologue and epilogue weigh more than the LDS
// traffic the larger wave tiles save (dense_full 379-396 against 350-364 us,
// dense_sub 87 against 76).
template <int BM, int WNN, int WMM>
constexpr size_t fuse_dma_lds_bytes() {
  return (size_t)2 * (BM + kMfmaBN) * kBK * 2 + (size_t)kMfmaBN * 4 + (size_t)2 * BM * 4 +
         (size_t)BM * 8;
}

template <int BM, int WNN, int WMM, bool O32>
__global__ __launch_bounds__(64 * WNN * WMM)
__attribute__((amdgpu_waves_per_eu(WNN * WMM / 4, WNN * WMM / 4)))
void k_fuse_dma(const MfmaArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int BN = kMfmaBN, NT = 64 * WNN * WMM;
  constexpr int FI = BN / WNN / 32, FJ = BM / WMM / 32;  // position / row fragments per wave
  static_assert(FI * WNN * 32 == BN && FJ * WMM * 32 == BM, "wave grid");
  constexpr int IW = 4;  // waves issuing the operand copies (one per SIMD)
  constexpr int A_INS = BM / 8 / IW, B_INS = BN / 8 / IW;
  static_assert(A_INS * 8 * IW == BM && B_INS * 8 * IW == BN, "copy instructions");
  constexpr int STAGE_B = (BM + BN) * kBK * 2;  // bytes of one operand stage
  constexpr bool kLastStep = BM * BN <= STAGE_B && BM <= BN;  // 8-bit tile fits in one stage
  extern __shared__ __align__(16) uint8_t smem[];
  uint16_t* As = reinterpret_cast<uint16_t*>(smem);                 // [2][BM][64]
  uint16_t* Bs = As + 2 * BM * kBK;                                  // [2][BN][64]
  int32_t* s_ids = reinterpret_cast<int32_t*>(smem + 2 * STAGE_B);
  float* s_sc = reinterpret_cast<float*>(s_ids + BN);               // [2][BM]: scale, dot factor
  unsigned long long* s_rkey = reinterpret_cast<unsigned long long*>(s_sc + 2 * BM);
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int iw = wave < IW ? wave : 0;
  const int wn = wave % WNN, wm = wave / WNN;
  int mt, nt;
  tile_of_block(blockIdx.x, a.m_tiles, a.n_tiles, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int M = a.M, K = a.K, n = a.n;
  const int last_id = a.ids[min(n, n0 + BN) - 1];
  for (int i = tid; i < BN; i += NT) s_ids[i] = n0 + i < n ? a.ids[n0 + i] : last_id;
  // a tile lies in one block of positions (blocks are multiples of BN)
  const int kb = a.qshift < 0 ? 0 : (n0 >> a.qshift);
  for (int i = tid; i < BM; i += NT) {
    s_rkey[i] = 0ull;
    s_sc[i] = m0 + i < M ? a.qscale[(int64_t)(m0 + i) * a.qnb + kb] : 0.0f;
    s_sc[BM + i] = (a.hscale && m0 + i < M) ? a.hscale[m0 + i] : 1.0f;
  }
  __syncthreads();
  const int lr = lane >> 3;
  const uint8_t* hbase = reinterpret_cast<const uint8_t*>(a.h);
  LaneAddr<O32> pa[A_INS], pb[B_INS];
#pragma unroll
  for (int i = 0; i < A_INS; ++i) {
    const int r = (iw * A_INS + i) * 8 + lr;
    const int lc = (lane & 7) ^ swz8(r);
    pa[i].set(hbase, (int64_t)min(m0 + r, M - 1) * a.ldh * 2 + lc * 16);
  }
#pragma unroll
  for (int i = 0; i < B_INS; ++i) {
    const int r = (iw * B_INS + i) * 8 + lr;
    const int lc = (lane & 7) ^ swz8(r);
    // weight row r of a 32-row group holds subset position pr: MFMA row
    // 8g + 4h + e (g = register group, h = lane / 32, e = element) gets
    // position 16h + 4g + e, so a lane's 16 accumulators cover 16
    // consecutive positions
    const int pr = (r & ~31) | (((r >> 2) & 1) << 4) | (((r >> 3) & 3) << 2) | (r & 3);
    pb[i].set(a.w, (int64_t)s_ids[pr] * a.ldw_bytes + lc * 16);
  }
  auto issue = [&](int k0, int stage) {
    if (wave >= IW) return;
    uint8_t* as = reinterpret_cast<uint8_t*>(As + stage * BM * kBK);
    uint8_t* bs = reinterpret_cast<uint8_t*>(Bs + stage * BN * kBK);
    const int64_t step = (int64_t)k0 * 2;
    const uint8_t* ha = O32 ? scalar_ptr(hbase + step) : nullptr;
    const uint8_t* wb = O32 ? scalar_ptr(a.w + step) : nullptr;
#pragma unroll
    for (int i = 0; i < A_INS; ++i) pa[i].copy(ha, step, (lds_void_t*)(as + (iw * A_INS + i) * 1024));
#pragma unroll
    for (int i = 0; i < B_INS; ++i) pb[i].copy(wb, step, (lds_void_t*)(bs + (iw * B_INS + i) * 1024));
  };
  const int qb = a.qbits;
  const int TB = BN * qb / 8;  // code bytes of a tile row
  const int CPR = TB / 16;     // 16-byte chunks of a tile row
  const int64_t c0 = (int64_t)n0 * qb / 8;
  const int64_t rowbytes = ((int64_t)n * qb + 7) / 8;
  const bool vec_q = (a.qstride & 15) == 0 && (reinterpret_cast<uintptr_t>(a.q) & 15) == 0;
  const bool dma_q = qb == 8 && vec_q;
  // chunk swizzle of payload row r: 16 chunks of 8-bit codes, 8 of 4-bit
  // codes (by r / 2, so that the 8-byte reads of 32 rows spread over the banks)
  auto qswz = [&](int r) { return qb == 8 ? (r & 15) : ((r >> 1) & 7); };
  // payload row r: staged in the last K step, rows [0, BM/2) in the idle
  // stage's A buffer and [BM/2, BM) in its B buffer; staged after the
  // loop, consecutive rows from the start of LDS
  auto prow = [&](bool in_stage, int st, int r) -> uint8_t* {
    if (!in_stage) return smem + r * TB;
    return r < BM / 2 ? reinterpret_cast<uint8_t*>(As + st * BM * kBK) + r * TB
                      : reinterpret_cast<uint8_t*>(Bs + st * BN * kBK) + (r - BM / 2) * TB;
  };
  // global-to-LDS copies of an 8-bit payload tile: a wave instruction fills
  // 4 rows (1 KB, contiguous in either placement); rows past M read row
  // M-1 and chunks past the row's end read the tile's first chunk (their
  // positions are never selected)
  auto stage_payload_dma = [&](bool in_stage, int st) {
    for (int t = wave; t < BM / 4; t += WNN * WMM) {
      const int r = t * 4 + (lane >> 4);
      const int k = (lane & 15) ^ (r & 15);
      const int64_t col = c0 + k * 16 < rowbytes ? c0 + k * 16 : c0;
      __builtin_amdgcn_global_load_lds(a.q + (int64_t)min(m0 + r, M - 1) * a.qstride + col,
                                       (lds_void_t*)prow(in_stage, st, t * 4), 16, 0, 0);
    }
  };

  f32x16_t acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  if (K > 0) {
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  int stage = 0;
  bool staged = false;
  for (int k0 = 0; k0 < K; k0 += kBK) {
    if (k0 + kBK < K) {
      issue(k0 + kBK, stage ^ 1);
    } else if (kLastStep && dma_q) {
      // the last step reads one stage; the payload tile goes to the other
      stage_payload_dma(true, stage ^ 1);
      staged = true;
    }
    const uint16_t* as = As + stage * BM * kBK;
    const uint16_t* bs = Bs + stage * BN * kBK;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8_t hf[FJ], wf[FI];
      const int c = kk * 2 + (lane >> 5);
#pragma unroll
      for (int j = 0; j < FJ; ++j) {
        const int row = wm * (BM / WMM) + j * 32 + (lane & 31);
        hf[j] = *reinterpret_cast<const bf16x8_t*>(as + row * kBK + ((c ^ swz8(row)) << 3));
      }
#pragma unroll
      for (int i = 0; i < FI; ++i) {
        const int row = wn * (BN / WNN) + i * 32 + (lane & 31);
        wf[i] = *reinterpret_cast<const bf16x8_t*>(bs + row * kBK + ((c ^ swz8(row)) << 3));
      }
#pragma unroll
      for (int i = 0; i < FI; ++i)
#pragma unroll
        for (int j = 0; j < FJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[i], hf[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies (operands or payload) have landed
    __syncthreads();
    stage ^= 1;
  }
  // after the last step's toggle, `stage` names the buffer that step did not read
  const int pst = stage;
  if (!staged) {
    if (dma_q) {
      stage_payload_dma(false, 0);
      __builtin_amdgcn_s_waitcnt(0);
    } else if (vec_q) {
      for (int c = tid; c < BM * CPR; c += NT) {
        const int r = c / CPR, k = c % CPR;
        const int64_t col = c0 + k * 16;
        const u32x4_t v = (m0 + r < M && col < rowbytes)
                              ? *reinterpret_cast<const u32x4_t*>(a.q + (int64_t)(m0 + r) * a.qstride + col)
                              : u32x4_t{0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4_t*>(prow(false, 0, r) + ((k ^ qswz(r)) << 4)) = v;
      }
    } else {
      for (int c = tid; c < BM * TB; c += NT) {
        const int r = c / TB, byte = c % TB, k = byte >> 4;
        const int64_t col = c0 + byte;
        prow(false, 0, r)[((k ^ qswz(r)) << 4) | (byte & 15)] =
            (m0 + r < M && col < rowbytes) ? a.q[(int64_t)(m0 + r) * a.qstride + col] : (uint8_t)0;
      }
    }
    __syncthreads();
  }
  // lane l of fragment (i, j) holds positions i*32 + 16*(l/32) + r of row
  // j*32 + l%32 in its 16 accumulators r: one 16-byte (8-bit) or 8-byte
  // (4-bit) LDS read gives the lane its codes; the lane's largest fused
  // value, then the lowest of its positions holding it
  const bool hq = a.hscale != nullptr;
  const int hh = lane >> 5;
  auto run = [&](auto edge, auto hidden) {
    constexpr bool kEdge = decltype(edge)::value;  // bounds checks and the fused output
    constexpr bool kHq = decltype(hidden)::value;  // rows carry hidden-state scales
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      const int ml = wm * (BM / WMM) + j * 32 + (lane & 31);
      const float sc = s_sc[ml];
      const uint8_t* qrow = prow(staged, pst, ml);
      u32x4_t cq[FI];
#pragma unroll
      for (int i = 0; i < FI; ++i) {
        const int nl0 = wn * (BN / WNN) + i * 32 + 16 * hh;
        if (qb == 8) {
          cq[i] = *reinterpret_cast<const u32x4_t*>(qrow + (((nl0 >> 4) ^ (ml & 15)) << 4));
        } else {
          const int bo = nl0 >> 1;
          const uint2 h2 = *reinterpret_cast<const uint2*>(qrow + ((((bo >> 4) ^ ((ml >> 1) & 7)) << 4) | (bo & 15)));
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const uint32_t h = ((g < 2 ? h2.x : h2.y) >> (16 * (g & 1))) & 0xFFFFu;
            uint32_t c4 = (h & 0xFu) | ((h & 0xF0u) << 4) | ((h & 0xF00u) << 8) | ((h & 0xF000u) << 12);
            c4 |= (c4 & 0x08080808u) * 0x1Eu;  // a nibble's sign bit fills bits 4..7 of its byte
            cq[i][g] = c4;
          }
        }
      }
      if constexpr (kHq) {
        const float hsc = s_sc[BM + ml];
#pragma unroll
        for (int i = 0; i < FI; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] *= hsc;
      }
      float bv = -__builtin_inff();
#pragma unroll
      for (int i = 0; i < FI; ++i) {
        const int nl0 = wn * (BN / WNN) + i * 32 + 16 * hh;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int code = (int)(int8_t)(cq[i][r >> 2] >> (8 * (r & 3)));
          acc[i][j][r] = __builtin_fmaf((float)code, sc, acc[i][j][r]);
        }
        if constexpr (kEdge) {
          if (a.f) {
            // lanes l and l + 32 trade halves so that each holds positions
            // 8q + 4*(l/32) + [0, 4) in registers 4*ro(q), ro = 0, 2, 1, 3:
            // each store instruction then covers 32 contiguous bytes of a row
            float x[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) x[r] = acc[i][j][r];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
#pragma unroll
              for (int b = 0; b < 16; b += 8) {
                const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[b + e]),
                                                                 __float_as_uint(x[b + 4 + e]), false, false);
                x[b + e] = __uint_as_float(sw[0]);
                x[b + 4 + e] = __uint_as_float(sw[1]);
              }
            }
            const int m = m0 + ml;
            if (m < M) {
              const int nlb = wn * (BN / WNN) + i * 32 + 4 * hh;
              float* dst = a.f + (int64_t)m * n + n0 + nlb;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int ro = ((q & 1) << 3) | ((q >> 1) << 2);
                if (n0 + nlb + 8 * q + 4 <= n && (reinterpret_cast<uintptr_t>(dst + 8 * q) & 15) == 0) {
                  *reinterpret_cast<float4*>(dst + 8 * q) = make_float4(x[ro], x[ro + 1], x[ro + 2], x[ro + 3]);
                } else {
#pragma unroll
                  for (int e = 0; e < 4; ++e)
                    if (n0 + nlb + 8 * q + e < n) dst[8 * q + e] = x[ro + e];
                }
              }
            }
          }
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (n0 + nl0 + r >= n) acc[i][j][r] = -__builtin_inff();
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) bv = fmaxf(bv, acc[i][j][r]);
      }
      int bn = 0;
#pragma unroll
      for (int t = FI * 16 - 1; t >= 0; --t) bn = acc[t >> 4][j][t & 15] == bv ? t : bn;
      const int pos = wn * (BN / WNN) + (bn >> 4) * 32 + 16 * hh + (bn & 15);
      unsigned long long key = bv > -__builtin_inff() ? argmax_key_m(bv, n0 + pos) : 0ull;
      const unsigned long long other = xor_lane_u64_32(key);
      key = key > other ? key : other;
      if (lane < 32) atomicMax(&s_rkey[ml], key);
    }
  };
  if (a.f || m0 + BM > M || n0 + BN > n) {
    if (hq) run(std::true_type{}, std::true_type{});
    else run(std::true_type{}, std::false_type{});
  } else {
    if (hq) run(std::false_type{}, std::true_type{});
    else run(std::false_type{}, std::false_type{});
  }
  __syncthreads();
  for (int i = tid; i < BM; i += NT)
    if (m0 + i < M) a.best_part[(int64_t)(m0 + i) * kMaxBlocks + nt] = s_rkey[i];
#endif
}

template <int BM, int BN>
constexpr size_t mfma_lds_bytes() {
  return (size_t)2 * (BM + BN) * kLDK * 2 + (size_t)BN * 4 + (size_t)(BM + 1) * 4 + 8 +
         (size_t)BM * 8;
}

template <int BM, int BN>
constexpr size_t mfma_dma_lds_bytes() {
  return (size_t)2 * (BM + BN) * kBK * 2 + (size_t)BN * 4 + (size_t)(BM + 1) * 4 + 8 +
         (size_t)BM * 8;
}

template <int BM, int BN>
constexpr size_t mfma_dma8_lds_bytes() {
  return (size_t)2 * (BM * 2 + BN) * kBK + (size_t)BN * 4 + (size_t)(BM + 1) * 4 + 8 +
         (size_t)BM * 8;
}

// Waves of a cloud row tile (the direct-to-LDS kernels).  256- and 320-row
// tiles use 8 waves, two per SIMD, so one wave's MFMAs run while the other
// waits at a barrier or on LDS: 2 x 4 (wave tiles 128 x 64 / 160 x 64),
// whose long K loop ran 6% faster so than with 4 x 2; on the dense 2048-row
// shape 8 waves ran 9% faster than 4 (wave tile 128 x 128).  128-row tiles
// use 2 x 2, 32-row tiles (9 to 32 rows) 1 x 4 waves of 32 x 64.  (The
// endpoint projection's transposed tiles choose their own grid.)
template <int BM, int EPI>
struct WaveGrid {
  static constexpr bool kEight = BM >= 256;
  static constexpr int WM = BM == 32 ? 1 : kEight ? 2 : 2;
  static constexpr int WN = BM == 32 ? 4 : kEight ? 4 : 2;
};

// The dynamic-LDS limit of a kernel is raised once per device (a host call,
// kept out of every launch so that launches can be captured in a graph).
// `done` is one instantiation's mask of devices already set.
static hipError_t set_lds_limit_once(std::atomic<uint64_t>& done, const void* kern, size_t bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? (uint64_t(1) << dev) : 0;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
  return e;
}

// 32-bit copy offsets (LaneAddr<true>) when every row the copies address
// lies below 4 GiB of its operand's base.
static bool copy_offsets_fit(const MfmaArgs& a) {
  constexpr int64_t kLim = 0xFFFFFFFFll;
  return a.w_rows > 0 && (int64_t)a.M * a.ldh * 2 <= kLim && a.w_rows * a.ldw_bytes <= kLim;
}

template <int BM, int BN, int WT, int EPI>
static hipError_t launch_tile(MfmaArgs a, hipStream_t s) {
  static std::atomic<uint64_t> lds_set_dma{0}, lds_set_dma64{0}, lds_set_reg{0};
  constexpr int WM = WaveGrid<BM, EPI>::WM, WN = WaveGrid<BM, EPI>::WN, NT = 64 * WM * WN;
  a.m_tiles = (a.M + BM - 1) / BM;
  a.n_tiles = (a.n + BN - 1) / BN;
  if (a.n_tiles > kMaxBlocks) return hipErrorInvalidValue;
  const bool o32 = copy_offsets_fit(a);
  if constexpr (EPI == kEpiFuse) {
    if (a.K % kBK == 0) {
      // transposed tiles: waves along the positions x waves along the rows
      constexpr int WNN = BM == 256 ? 2 : BM == 320 ? 4 : BM == 128 ? 2 : 4;
      constexpr int WMM = BM == 256 ? 4 : BM == 320 ? 2 : BM == 128 ? 2 : 1;
      auto kf = o32 ? k_fuse_dma<BM, WNN, WMM, true> : k_fuse_dma<BM, WNN, WMM, false>;
      constexpr size_t lds_f = fuse_dma_lds_bytes<BM, WNN, WMM>();
      static std::atomic<uint64_t> lds_set_fuse{0}, lds_set_fuse64{0};
      hipError_t e = set_lds_limit_once(o32 ? lds_set_fuse : lds_set_fuse64,
                                        reinterpret_cast<const void*>(kf), lds_f);
      if (e != hipSuccess) return e;
      launch_kernel(kf, dim3(a.m_tiles * a.n_tiles), dim3(64 * WNN * WMM), lds_f, s, a);
      return hipGetLastError();
    }
  } else if (a.K % kBK == 0) {
    if constexpr (BM == 256 && WT == 0 && EPI == kEpiCloud) {
      // (the one-wave kernels copy their first steps unconditionally: they
      // need at least 6 or 2 steps; a zero-width slice takes the kernel below)
      if (o32 && a.K >= 6 * kBK && (a.K / kBK) % 6 == 0) {
        // one wave per SIMD, three weight stages (all 160 KB of LDS)
        static std::atomic<uint64_t> lds_set_w3{0};
        constexpr size_t lds_w = (size_t)5 * BM * kBK * 2;
        hipError_t e = set_lds_limit_once(lds_set_w3, reinterpret_cast<const void*>(k_mfma_w1<EPI, 3>), lds_w);
        if (e != hipSuccess) return e;
        launch_kernel(k_mfma_w1<EPI, 3>, dim3(a.m_tiles * a.n_tiles), dim3(256), lds_w, s, a);
        return hipGetLastError();
      }
      if (o32 && a.K >= 2 * kBK && (a.K / kBK) % 2 == 0) {
        // one wave per SIMD (an even number of K steps)
        static std::atomic<uint64_t> lds_set_w1{0};
        constexpr size_t lds_w = mfma_dma_lds_bytes<BM, BN>();
        hipError_t e = set_lds_limit_once(lds_set_w1, reinterpret_cast<const void*>(k_mfma_w1<EPI, 2>), lds_w);
        if (e != hipSuccess) return e;
        launch_kernel(k_mfma_w1<EPI, 2>, dim3(a.m_tiles * a.n_tiles), dim3(256), lds_w, s, a);
        return hipGetLastError();
      }
    }
    auto kd = WT == 0 ? (o32 ? k_mfma_dma<BM, BN, WM, WN, EPI, true> : k_mfma_dma<BM, BN, WM, WN, EPI, false>)
                      : (o32 ? k_mfma_dma8<BM, BN, WM, WN, EPI, true> : k_mfma_dma8<BM, BN, WM, WN, EPI, false>);
    constexpr size_t lds_d = WT == 0 ? mfma_dma_lds_bytes<BM, BN>() : mfma_dma8_lds_bytes<BM, BN>();
    hipError_t e = set_lds_limit_once(o32 ? lds_set_dma : lds_set_dma64, reinterpret_cast<const void*>(kd), lds_d);
    if (e != hipSuccess) return e;
    launch_kernel(kd, dim3(a.m_tiles * a.n_tiles), dim3(NT), lds_d, s, a);
    return hipGetLastError();
  }
  // K not a multiple of the K step: the register-staged kernel (2 x 2 waves),
  // which exists for 128- and 256-row tiles (the tile rule picks neither 32
  // nor 320 then)
  if constexpr (BM >= 128 && BM <= 256 && EPI != kEpiCloudQ) {
    auto kern = k_mfma<BM, BN, WT, EPI>;
    constexpr size_t lds = mfma_lds_bytes<BM, BN>();
    hipError_t e = set_lds_limit_once(lds_set_reg, reinterpret_cast<const void*>(kern), lds);
    if (e != hipSuccess) return e;
    launch_kernel(kern, dim3(a.m_tiles * a.n_tiles), dim3(256), lds, s, a);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

// Row tile for M rows: 32 up to 32 rows (K a multiple of the K step), 128
// up to 128 rows, else whichever of 256 and 320
// pads M less (320-row tiles need K a multiple of the K step).  Measured on
// the batched shape (M = 320, 60000 ids): 320-row tiles, one per 256 ids,
// 156 us against 265 us for 256-row and 289 us for 128-row tiles; M = 640
// with fp8 weights: 460 us against 537 us for 256-row tiles.
static int mfma_bm(int M, int K) {
  // up to 32 rows the projection streams its weights like the skinny kernel
  // does; a 32-row tile wastes at most 23 of 32 rows of MFMA work instead of
  // 119 of 128, and two blocks fit on a CU
  if (M <= 32 && K % kBK == 0) return 32;
  if (M <= 128) return 128;
  const int pad256 = (M + 255) / 256 * 256 - M;
  const int pad320 = (M + 319) / 320 * 320 - M;
  return (K % kBK == 0 && pad320 < pad256) ? 320 : 256;
}

int mfma_n_tiles(int n) { return (n + kMfmaBN - 1) / kMfmaBN; }

template <int WT, int EPI>
static hipError_t launch_bm(const MfmaArgs& a, hipStream_t s) {
  switch (mfma_bm(a.M, a.K)) {
    case 32: return launch_tile<32, kMfmaBN, WT, EPI>(a, s);
    case 320: return launch_tile<320, kMfmaBN, WT, EPI>(a, s);
    case 256: return launch_tile<256, kMfmaBN, WT, EPI>(a, s);
    default: return launch_tile<128, kMfmaBN, WT, EPI>(a, s);
  }
}

// Cloud projection with the block quantiser in the epilogue, for the row
// tiles whose accumulators and row maxima fit in the registers together
// (32, 128, 256 rows, K a multiple of the K step).  Where the tile rule picks
// 320 rows the separate quantiser is used: on 640 rows, 256-row tiles with
// the fused quantiser ran 598 us against 428 + 43 us.
bool mfma_quantises_in_epilogue(int M, int K) {
  return K % kBK == 0 && mfma_bm(M, K) != 320;
}

template <int WT>
static hipError_t launch_bm_q(const MfmaArgs& a, hipStream_t s) {
  if (!mfma_quantises_in_epilogue(a.M, a.K)) return hipErrorInvalidValue;
  switch (mfma_bm(a.M, a.K)) {
    case 32: return launch_tile<32, kMfmaBN, WT, kEpiCloudQ>(a, s);
    case 128: return launch_tile<128, kMfmaBN, WT, kEpiCloudQ>(a, s);
    default: return launch_tile<256, kMfmaBN, WT, kEpiCloudQ>(a, s);
  }
}

hipError_t launch_mfma(int epi, int wtype, const MfmaArgs& a, hipStream_t s) {
  if (epi == kEpiCloudQ) return wtype == 0 ? launch_bm_q<0>(a, s) : launch_bm_q<1>(a, s);
  if (epi == kEpiCloud)
    return wtype == 0 ? launch_bm<0, kEpiCloud>(a, s) : launch_bm<1, kEpiCloud>(a, s);
  if (wtype != 0) return hipErrorInvalidValue;
  return launch_bm<0, kEpiFuse>(a, s);
}

}  // namespace sph
