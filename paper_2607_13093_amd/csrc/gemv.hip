// Skinny gathered projection for few rows of h (VALU path, HBM bound).
//
// Computes, for every subset position j and every row m of one launch,
//   acc[m, j] = sum_i h[m, i] * W[S_j, i]
// which is eq. 12 for the cloud slice and eq. 11 for the endpoint slice
// (Section 5.4), both restricted to the language subset S.  With only a
// handful of rows the work is a stream over the gathered weight rows: every
// weight byte is read once from HBM and used for every row of h.
//
// Layout of the work:
//  * Each block owns a contiguous range of subset positions.  The rows of h
//    (bf16, zero padded to whole weight chunks) and the block's subset ids
//    are staged once in LDS.
//  * A group of LPR lanes owns one vocabulary row at a time; lane c of the
//    group reads 16-byte chunks c, c + LPR, ... of the row, so one load
//    instruction of a wave covers LPR contiguous chunks of 64/LPR rows.
//    Each lane issues UNR (4 or 8) such loads before using any of them, and
//    the loads are non-temporal: every weight byte is used exactly once.
//  * 512-thread blocks share one staged copy of h, so LDS does not cap the
//    number of resident waves; the kernel is built for at least 4 waves per
//    SIMD (at most 128 VGPRs).  A register double buffer and two rows per
//    lane group were measured slower: they cost waves, not latency.
//  * bf16 products use v_dot2_f32_bf16 (two products and one fp32 add per
//    instruction, fp32 accumulation); fp8 E4M3 chunks are widened to bf16
//    in registers first (exact: every E4M3 value is a bf16 value).
//  * The VR x MR sums of a group are reduced across its LPR lanes by a
//    transposing butterfly: each exchange halves the number of values a lane
//    carries, so the reduction costs about VR*MR exchanges instead of
//    VR*MR*log2(LPR).
//  * Epilogues: the cloud epilogue scales fp8 rows, adds the bias, writes the
//    fp32 partial logit and keeps a running max of |clamp(z)| per row; the
//    fuse epilogue dequantises the payload (eq. 13), writes the fused logit
//    on request and keeps a running (value, position) argmax per row.  Both
//    are folded per block into partial slots read by the row-wide kernels.
#include "sph_internal.h"

namespace sph {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// Two E4M3 bytes (selected half of x) -> two bf16 in one word, exact.
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_to_bf16x2(uint32_t x) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, HI));
}

// Orderable 64-bit key: larger value first, then the lower position.
__device__ __forceinline__ unsigned long long argmax_key(float v, int pos) {
  v = v + 0.0f;  // -0 -> +0 so that equal values compare equal
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)u << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)pos);
}

constexpr int pow2ceil(int x) { return x <= 1 ? 1 : 2 * pow2ceil((x + 1) / 2); }
constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

// Transposing butterfly over the LPR lanes of a group.  On return, if
// P <= LPR, lane c of the group holds the total of value c >> (log2 LPR -
// log2 P) in v[0]; otherwise it holds values c*P/LPR .. (c+1)*P/LPR - 1.
template <int P, int LPR>
__device__ __forceinline__ void xreduce(float (&v)[P], int lane) {
  int cnt = P;
#pragma unroll
  for (int o = LPR / 2; o >= 1; o >>= 1) {
    if (cnt > 1) {
      const int half = cnt / 2;
      const bool upper = (lane & o) != 0;
#pragma unroll
      for (int i = 0; i < half; ++i) {
        const float send = upper ? v[i] : v[i + half];
        const float keep = upper ? v[i + half] : v[i];
        v[i] = keep + __shfl_xor(send, o, 64);
      }
      cnt = half;
    } else {
      v[0] += __shfl_xor(v[0], o, 64);
    }
  }
}

constexpr int kVR = 1;    // vocabulary rows per lane group in flight
constexpr int kBS = 512;  // threads per block

template <int LPR>
struct GemvShape {
  static constexpr int GPW = 64 / LPR;                   // lane groups per wave
  static constexpr int RPI = (kBS / 64) * GPW * kVR;     // rows per block iteration
};

template <int MR, int LPR, int UNR, int WT, int EPI>
__global__ __launch_bounds__(kBS) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_gemv(const GemvArgs a) {
  constexpr int VR = kVR;
  constexpr int GPW = GemvShape<LPR>::GPW, RPI = GemvShape<LPR>::RPI;
  constexpr int EPC = WT == 0 ? 8 : 16;  // weight elements per 16-byte chunk
  constexpr int HW = EPC / 2;            // h words (bf16 pairs) per chunk
  constexpr int NV = VR * MR;
  constexpr int P = pow2ceil(NV);
  constexpr int PER = P > LPR ? P / LPR : 1;

  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ uint32_t s_amax[MR];
  __shared__ unsigned long long s_best[MR];

  const int Kp = a.Kp;
  uint16_t* hs = reinterpret_cast<uint16_t*>(smem);
  int32_t* s_ids = reinterpret_cast<int32_t*>(smem + (size_t)MR * Kp * 2);
  const int tid = threadIdx.x;
  const int n = a.n;
  const int r0 = blockIdx.x * a.rows_per_block;
  const int r1 = min(n, r0 + a.rows_per_block);

  if (tid < MR) {
    s_amax[tid] = 0u;
    s_best[tid] = 0ull;
  }
  // Stage h[0:MR, 0:K] into LDS, zero padded to Kp, and this block's ids.
  if ((reinterpret_cast<uintptr_t>(a.h) & 15) == 0 && (a.ldh & 7) == 0 && (a.K & 7) == 0) {
    const int vpr = Kp / 8;  // 16-byte vectors per staged row
    for (int idx = tid; idx < MR * vpr; idx += kBS) {
      const int m = idx / vpr, c = idx - m * vpr;
      u32x4_t val = {0u, 0u, 0u, 0u};
      if (c * 8 < a.K) val = *reinterpret_cast<const u32x4_t*>(a.h + (int64_t)m * a.ldh + c * 8);
      *reinterpret_cast<u32x4_t*>(hs + m * Kp + c * 8) = val;
    }
  } else {
    for (int idx = tid; idx < MR * Kp; idx += kBS) {
      const int m = idx / Kp, k = idx - m * Kp;
      hs[idx] = k < a.K ? a.h[(int64_t)m * a.ldh + k] : (uint16_t)0;
    }
  }
  for (int j = r0 + tid; j < r1; j += kBS) s_ids[j - r0] = a.ids[j];
  __syncthreads();

  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int cl = lane % LPR;
  const int grp = wave * GPW + lane / LPR;
  const int nchunk = Kp / EPC;

  // Which reduced values this lane ends up holding (fixed for the whole
  // kernel): value i is (row v = own_idx / MR of the group, h row m = own_idx % MR).
  int own_idx[PER];
  bool own[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if constexpr (P > LPR) {
      own_idx[i] = cl * PER + i;
      own[i] = own_idx[i] < NV;
    } else {
      constexpr int sh = ilog2(LPR) - ilog2(P);
      own_idx[i] = cl >> sh;
      own[i] = (cl & ((1 << sh) - 1)) == 0 && own_idx[i] < NV;
    }
  }
  float run_amax[PER];
  unsigned long long run_key[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    run_amax[i] = 0.0f;
    run_key[i] = 0ull;
  }

  // Flat item stream: item t = (iteration t / passes, pass t % passes).
  const int passes = nchunk > 0 ? (nchunk + LPR * UNR - 1) / (LPR * UNR) : 1;
  const int iters = (r1 - r0 + RPI - 1) / RPI;
  const int T = r1 > r0 ? iters * passes : 0;

  u32x4_t cur[UNR][VR];
  int qcur[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) qcur[i] = 0;

  auto load_item = [&](int t, u32x4_t (&buf)[UNR][VR], int (&qb)[PER]) {
    const int it = t / passes, pass = t - it * passes;
    const int jb = r0 + it * RPI + grp * VR;
#pragma unroll
    for (int v = 0; v < VR; ++v) {
      const int j = jb + v;
      const bool ok = j < r1;
      const uint8_t* row = a.w + (int64_t)(ok ? s_ids[j - r0] : 0) * a.ldw_bytes;
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int c = cl + (pass * UNR + u) * LPR;
        if (ok && c < nchunk)
          buf[u][v] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(row + (int64_t)c * 16));
        else
          buf[u][v] = u32x4_t{0u, 0u, 0u, 0u};
      }
    }
    if constexpr (EPI == kEpiFuse) {
      if (pass == 0) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
          const int j = jb + own_idx[i] / MR;
          qb[i] = (own[i] && j < r1) ? (int)a.q[(int64_t)(own_idx[i] % MR) * n + j] : 0;
        }
      }
    }
  };

  float acc[VR][MR];
#pragma unroll
  for (int v = 0; v < VR; ++v)
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[v][m] = 0.0f;

  for (int t = 0; t < T; ++t) {
    const int it = t / passes, pass = t - it * passes;
    load_item(t, cur, qcur);

#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int c = cl + (pass * UNR + u) * LPR;
      if (c < nchunk) {
#pragma unroll
        for (int m = 0; m < MR; ++m) {
          const uint32_t* hp = reinterpret_cast<const uint32_t*>(hs + m * Kp + c * EPC);
          uint32_t hw[HW];
#pragma unroll
          for (int e = 0; e < HW; e += 4) {
            const u32x4_t x = *reinterpret_cast<const u32x4_t*>(hp + e);
            hw[e] = x.x; hw[e + 1] = x.y; hw[e + 2] = x.z; hw[e + 3] = x.w;
          }
#pragma unroll
          for (int v = 0; v < VR; ++v) {
            float s = acc[v][m];
            if constexpr (WT == 0) {
              s = dot2_bf16(cur[u][v].x, hw[0], s);
              s = dot2_bf16(cur[u][v].y, hw[1], s);
              s = dot2_bf16(cur[u][v].z, hw[2], s);
              s = dot2_bf16(cur[u][v].w, hw[3], s);
            } else {
              const uint32_t w4[4] = {cur[u][v].x, cur[u][v].y, cur[u][v].z, cur[u][v].w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                s = dot2_bf16(e4m3x2_to_bf16x2<false>(w4[e]), hw[2 * e], s);
                s = dot2_bf16(e4m3x2_to_bf16x2<true>(w4[e]), hw[2 * e + 1], s);
              }
            }
            acc[v][m] = s;
          }
        }
      }
    }

    if (pass == passes - 1) {
      float vals[P];
#pragma unroll
      for (int i = 0; i < P; ++i) vals[i] = i < NV ? acc[i / MR][i % MR] : 0.0f;
      xreduce<P, LPR>(vals, lane);
      const int jb = r0 + it * RPI + grp * VR;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int m = own_idx[i] % MR;
        const int j = jb + own_idx[i] / MR;
        if (!own[i] || j >= r1) continue;
        const float dot = vals[i];
        if constexpr (EPI == kEpiCloud) {
          float z = dot;
          if constexpr (WT == 1) z = z * a.wscale[s_ids[j - r0]];
          if (a.bias) z = z + a.bias[s_ids[j - r0]];
          a.z[(int64_t)m * n + j] = z;
          const float y = fminf(fmaxf(z, -a.clip), a.clip);
          run_amax[i] = fmaxf(run_amax[i], fabsf(y));
        } else {
          const float f = __builtin_fmaf((float)qcur[i], a.qscale[m], dot);
          if (a.f) a.f[(int64_t)m * n + j] = f;
          const unsigned long long key = argmax_key(f, j);
          run_key[i] = key > run_key[i] ? key : run_key[i];
        }
      }
#pragma unroll
      for (int v = 0; v < VR; ++v)
#pragma unroll
        for (int m = 0; m < MR; ++m) acc[v][m] = 0.0f;
    }
  }

#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (!own[i]) continue;
    const int m = own_idx[i] % MR;
    if constexpr (EPI == kEpiCloud)
      atomicMax(&s_amax[m], __float_as_uint(run_amax[i]));
    else
      atomicMax(&s_best[m], run_key[i]);
  }
  __syncthreads();
  // Block b owns partial slot b and zero-fills slots b + gridDim.x, ... below
  // a.nblk, so the consumer can fold a.nblk slots whatever the grid size.
  if (tid < MR) {
    for (int b = blockIdx.x; b < a.nblk; b += gridDim.x) {
      const bool mine = b == (int)blockIdx.x;
      if constexpr (EPI == kEpiCloud)
        a.amax_part[(int64_t)tid * kMaxBlocks + b] = mine ? __uint_as_float(s_amax[tid]) : 0.0f;
      else
        a.best_part[(int64_t)tid * kMaxBlocks + b] = mine ? s_best[tid] : 0ull;
    }
  }
}

// Lanes per vocabulary row: enough that each lane loads about four 16-byte
// chunks of the row, so short rows (the endpoint slice) are not spread over
// a whole wave and reduced across 64 lanes.
int gemv_lpr(int K, int wtype) {
  const int epc = wtype == 0 ? 8 : 16;
  const int chunks = (K + epc - 1) / epc;
  int lpr = 8;
  while (lpr < 64 && lpr * 4 < chunks) lpr *= 2;
  return lpr;
}

int gemv_rows_per_iter(int lpr) { return 4 * (64 / lpr) * kVR; }

// Chunks per lane per pass.
static int gemv_unr(int K, int wtype, int lpr) {
  const int epc = wtype == 0 ? 8 : 16;
  const int chunks = (K + epc - 1) / epc;
  const int per_lane = (chunks + lpr - 1) / lpr;
  return per_lane <= 4 ? 4 : 8;
}

template <int MR, int LPR, int UNR, int WT, int EPI>
static hipError_t launch_one(GemvArgs a, hipStream_t s) {
  auto kern = k_gemv<MR, LPR, UNR, WT, EPI>;
  const size_t hbytes = (size_t)MR * a.Kp * 2;
  constexpr int rpi = GemvShape<LPR>::RPI;
  const int iters = (a.n + rpi - 1) / rpi;
  // One round of resident blocks where possible: each block takes an equal
  // contiguous share of the subset positions.
  int resident = kMaxBlocks;
  int per_cu = 0, dev = 0, cus = 0;
  const size_t lds_guess = hbytes + 512 * 4;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kBS, lds_guess) == hipSuccess &&
      per_cu > 0 && cus > 0)
    resident = per_cu * cus;
  int grid = iters < resident ? iters : resident;
  if (grid > a.nblk) grid = a.nblk;
  int ipb = (iters + grid - 1) / grid;  // iterations per block
  if (ipb * rpi > kGemvMaxIdsPerBlock) ipb = kGemvMaxIdsPerBlock / rpi;  // more rounds instead
  if ((int64_t)ipb * rpi * a.nblk < a.n) return hipErrorInvalidValue;
  a.rows_per_block = ipb * rpi;
  grid = (a.n + a.rows_per_block - 1) / a.rows_per_block;
  const size_t lds = hbytes + (size_t)a.rows_per_block * 4;
  launch_kernel(kern, dim3(grid), dim3(kBS), lds, s, a);
  return hipGetLastError();
}

template <int LPR, int UNR, int WT, int EPI>
static hipError_t launch_rows(int rows, const GemvArgs& a, hipStream_t s) {
  switch (rows) {
    case 1: return launch_one<1, LPR, UNR, WT, EPI>(a, s);
    case 2: return launch_one<2, LPR, UNR, WT, EPI>(a, s);
    case 3: return launch_one<3, LPR, UNR, WT, EPI>(a, s);
    case 4: return launch_one<4, LPR, UNR, WT, EPI>(a, s);
    case 5: return launch_one<5, LPR, UNR, WT, EPI>(a, s);
    case 6: return launch_one<6, LPR, UNR, WT, EPI>(a, s);
    case 7: return launch_one<7, LPR, UNR, WT, EPI>(a, s);
    case 8: return launch_one<8, LPR, UNR, WT, EPI>(a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int LPR, int WT, int EPI>
static hipError_t launch_unr(int unr, int rows, const GemvArgs& a, hipStream_t s) {
  return unr == 4 ? launch_rows<LPR, 4, WT, EPI>(rows, a, s) : launch_rows<LPR, 8, WT, EPI>(rows, a, s);
}

template <int WT, int EPI>
static hipError_t launch_lpr(int lpr, int unr, int rows, const GemvArgs& a, hipStream_t s) {
  switch (lpr) {
    case 8: return launch_unr<8, WT, EPI>(unr, rows, a, s);
    case 16: return launch_unr<16, WT, EPI>(unr, rows, a, s);
    case 32: return launch_unr<32, WT, EPI>(unr, rows, a, s);
    case 64: return launch_unr<64, WT, EPI>(unr, rows, a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemv(int epi, int wtype, int rows, const GemvArgs& a, hipStream_t s) {
  const int lpr = gemv_lpr(a.K, wtype);
  const int unr = gemv_unr(a.K, wtype, lpr);
  if (epi == kEpiCloud)
    return wtype == 0 ? launch_lpr<0, kEpiCloud>(lpr, unr, rows, a, s)
                      : launch_lpr<1, kEpiCloud>(lpr, unr, rows, a, s);
  if (wtype != 0) return hipErrorInvalidValue;
  return launch_lpr<0, kEpiFuse>(lpr, unr, rows, a, s);
}

}  // namespace sph
