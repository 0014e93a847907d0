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
//  * The rows of h (bf16) are staged once per block in LDS, zero padded to a
//    whole number of weight chunks.
//  * A group of LPR lanes owns one vocabulary row at a time; lane c of the
//    group reads 16-byte chunks c, c + LPR, ... of that row, so each load
//    instruction of a wave covers 64 contiguous 16-byte chunks (1 KB) of
//    weight rows.  Each lane keeps VR rows in flight with UNR chunks each.
//  * bf16 products use v_dot2_f32_bf16 (two products and one fp32 add per
//    instruction, fp32 accumulation); fp8 E4M3 chunks are widened to bf16
//    in registers first (exact: every E4M3 value is a bf16 value).
//  * The VR x MR partial sums of a group are reduced across its LPR lanes by
//    a transposing butterfly: each exchange halves the number of values a
//    lane carries, so the reduction costs about VR*MR exchanges instead of
//    VR*MR*log2(LPR).
//  * Epilogues: the cloud epilogue scales fp8 rows, adds the bias, writes the
//    fp32 partial logit and folds |clamp(z)| into a per-block row maximum;
//    the fuse epilogue dequantises the payload (eq. 13), writes the fused
//    logit on request and folds (value, position) into a per-block argmax.
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
__device__ __forceinline__ uint64_t argmax_key(float v, int pos) {
  v = v + 0.0f;  // -0 -> +0 so that equal values compare equal
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)pos);
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

template <int EPI, int LPR>
struct GemvShape {
  static constexpr int VR = EPI == kEpiCloud ? 2 : 4;   // rows in flight per lane group
  static constexpr int UNR = EPI == kEpiCloud ? 4 : 2;  // chunks in flight per row
  static constexpr int GPW = 64 / LPR;                  // lane groups per wave
  static constexpr int RPI = 4 * GPW * VR;              // rows per block iteration
};

template <int MR, int LPR, int WT, int EPI>
__global__ __launch_bounds__(256) void k_gemv(const GemvArgs a) {
  using Sh = GemvShape<EPI, LPR>;
  constexpr int VR = Sh::VR, UNR = Sh::UNR, GPW = Sh::GPW, RPI = Sh::RPI;
  constexpr int EPC = WT == 0 ? 8 : 16;       // weight elements per 16-byte chunk
  constexpr int HW = EPC / 2;                 // h words (bf16 pairs) per chunk
  constexpr int NV = VR * MR;
  constexpr int P = pow2ceil(NV);

  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ uint32_t s_amax[MR];
  __shared__ unsigned long long s_best[MR];

  const int Kp = a.Kp;
  uint16_t* hs = reinterpret_cast<uint16_t*>(smem);
  const int tid = threadIdx.x;

  if (tid < MR) {
    s_amax[tid] = 0u;
    s_best[tid] = 0ull;
  }
  // Stage h[0:MR, 0:K] into LDS, zero padded to Kp.
  if ((reinterpret_cast<uintptr_t>(a.h) & 15) == 0 && (a.ldh & 7) == 0 && (a.K & 7) == 0) {
    const int vpr = Kp / 8;  // 16-byte vectors per staged row
    for (int idx = tid; idx < MR * vpr; idx += 256) {
      const int m = idx / vpr, c = idx - m * vpr;
      u32x4_t val = {0u, 0u, 0u, 0u};
      if (c * 8 < a.K) val = *reinterpret_cast<const u32x4_t*>(a.h + (int64_t)m * a.ldh + c * 8);
      *reinterpret_cast<u32x4_t*>(hs + m * Kp + c * 8) = val;
    }
  } else {
    for (int idx = tid; idx < MR * Kp; idx += 256) {
      const int m = idx / Kp, k = idx - m * Kp;
      hs[idx] = k < a.K ? a.h[(int64_t)m * a.ldh + k] : (uint16_t)0;
    }
  }
  __syncthreads();

  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int cl = lane % LPR;
  const int grp = wave * GPW + lane / LPR;
  const int nchunk = Kp / EPC;
  const int n = a.n;

  for (int base = blockIdx.x * RPI; base < n; base += gridDim.x * RPI) {
    const uint8_t* wrow[VR];
    bool valid[VR];
#pragma unroll
    for (int v = 0; v < VR; ++v) {
      const int j = base + grp * VR + v;
      valid[v] = j < n;
      const int id = valid[v] ? a.ids[j] : 0;
      wrow[v] = a.w + (int64_t)id * a.ldw_bytes;
    }
    float acc[VR][MR];
#pragma unroll
    for (int v = 0; v < VR; ++v)
#pragma unroll
      for (int m = 0; m < MR; ++m) acc[v][m] = 0.0f;

    for (int c0 = cl; c0 < nchunk; c0 += LPR * UNR) {
      u32x4_t wv[UNR][VR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int c = c0 + u * LPR;
#pragma unroll
        for (int v = 0; v < VR; ++v) {
          if (c < nchunk && valid[v])
            wv[u][v] = *reinterpret_cast<const u32x4_t*>(wrow[v] + (int64_t)c * 16);
          else
            wv[u][v] = u32x4_t{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int c = c0 + u * LPR;
        if (c < nchunk) {
#pragma unroll
          for (int m = 0; m < MR; ++m) {
            const uint32_t* hp = reinterpret_cast<const uint32_t*>(hs + m * Kp + c * EPC);
            uint32_t hw[HW];
#pragma unroll
            for (int t = 0; t < HW; t += 4) {
              const u32x4_t x = *reinterpret_cast<const u32x4_t*>(hp + t);
              hw[t] = x.x; hw[t + 1] = x.y; hw[t + 2] = x.z; hw[t + 3] = x.w;
            }
#pragma unroll
            for (int v = 0; v < VR; ++v) {
              float s = acc[v][m];
              if constexpr (WT == 0) {
                s = dot2_bf16(wv[u][v].x, hw[0], s);
                s = dot2_bf16(wv[u][v].y, hw[1], s);
                s = dot2_bf16(wv[u][v].z, hw[2], s);
                s = dot2_bf16(wv[u][v].w, hw[3], s);
              } else {
                const uint32_t q4[4] = {wv[u][v].x, wv[u][v].y, wv[u][v].z, wv[u][v].w};
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                  s = dot2_bf16(e4m3x2_to_bf16x2<false>(q4[t]), hw[2 * t], s);
                  s = dot2_bf16(e4m3x2_to_bf16x2<true>(q4[t]), hw[2 * t + 1], s);
                }
              }
              acc[v][m] = s;
            }
          }
        }
      }
    }

    float vals[P];
#pragma unroll
    for (int i = 0; i < P; ++i) vals[i] = i < NV ? acc[i / MR][i % MR] : 0.0f;
    xreduce<P, LPR>(vals, lane);

    constexpr int PER = P > LPR ? P / LPR : 1;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int idx;
      bool owner;
      if constexpr (P > LPR) {
        idx = cl * PER + i;
        owner = true;
      } else {
        constexpr int sh = ilog2(LPR) - ilog2(P);
        idx = cl >> sh;
        owner = (cl & ((1 << sh) - 1)) == 0;
      }
      if (!owner || idx >= NV) continue;
      const int v = idx / MR, m = idx % MR;
      const int j = base + grp * VR + v;
      if (j >= n) continue;
      const float dot = vals[i];
      if constexpr (EPI == kEpiCloud) {
        const int id = a.ids[j];
        float z = dot;
        if constexpr (WT == 1) z = z * a.wscale[id];
        if (a.bias) z = z + a.bias[id];
        a.z[(int64_t)m * n + j] = z;
        const float y = fminf(fmaxf(z, -a.clip), a.clip);
        atomicMax(&s_amax[m], __float_as_uint(fabsf(y)));
      } else {
        const float f = __builtin_fmaf((float)a.q[(int64_t)m * n + j], a.qscale[m], dot);
        if (a.f) a.f[(int64_t)m * n + j] = f;
        atomicMax(&s_best[m], (unsigned long long)argmax_key(f, j));
      }
    }
  }
  __syncthreads();
  if (tid < MR) {
    if constexpr (EPI == kEpiCloud)
      a.amax_part[(int64_t)tid * kMaxBlocks + blockIdx.x] = __uint_as_float(s_amax[tid]);
    else
      a.best_part[(int64_t)tid * kMaxBlocks + blockIdx.x] = s_best[tid];
  }
}

int gemv_rows_per_iter(int epi, int lpr) {
  const int vr = epi == kEpiCloud ? GemvShape<kEpiCloud, 64>::VR : GemvShape<kEpiFuse, 64>::VR;
  return 4 * (64 / lpr) * vr;
}

int gemv_lpr(int epi, int K, int wtype) {
  if (epi == kEpiCloud) return 64;
  const int epc = wtype == 0 ? 8 : 16;
  const int chunks = (K + epc - 1) / epc;
  int lpr = 8;
  while (lpr < 64 && lpr < chunks) lpr *= 2;
  return lpr;
}

template <int MR, int LPR, int WT, int EPI>
static hipError_t launch_one(const GemvArgs& a, hipStream_t s) {
  const size_t lds = (size_t)MR * a.Kp * 2;
  hipLaunchKernelGGL((k_gemv<MR, LPR, WT, EPI>), dim3(a.nblk), dim3(256), lds, s, a);
  return hipGetLastError();
}

template <int LPR, int WT, int EPI>
static hipError_t launch_rows(int rows, const GemvArgs& a, hipStream_t s) {
  switch (rows) {
    case 1: return launch_one<1, LPR, WT, EPI>(a, s);
    case 2: return launch_one<2, LPR, WT, EPI>(a, s);
    case 3: return launch_one<3, LPR, WT, EPI>(a, s);
    case 4: return launch_one<4, LPR, WT, EPI>(a, s);
    case 5: return launch_one<5, LPR, WT, EPI>(a, s);
    case 6: return launch_one<6, LPR, WT, EPI>(a, s);
    case 7: return launch_one<7, LPR, WT, EPI>(a, s);
    case 8: return launch_one<8, LPR, WT, EPI>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemv(int epi, int wtype, int rows, int lpr, const GemvArgs& a, hipStream_t s) {
  if (epi == kEpiCloud) {
    if (lpr != 64) return hipErrorInvalidValue;
    return wtype == 0 ? launch_rows<64, 0, kEpiCloud>(rows, a, s)
                      : launch_rows<64, 1, kEpiCloud>(rows, a, s);
  }
  if (wtype != 0) return hipErrorInvalidValue;
  switch (lpr) {
    case 8: return launch_rows<8, 0, kEpiFuse>(rows, a, s);
    case 16: return launch_rows<16, 0, kEpiFuse>(rows, a, s);
    case 32: return launch_rows<32, 0, kEpiFuse>(rows, a, s);
    case 64: return launch_rows<64, 0, kEpiFuse>(rows, a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sph
