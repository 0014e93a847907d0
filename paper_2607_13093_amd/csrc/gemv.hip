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
// Global-memory views of weight rows (loads through them are global, not flat).
typedef __attribute__((address_space(1))) const uint8_t gbyte;
typedef __attribute__((address_space(1))) const u32x4_t gu32x4;
// Constant-space view: a load through it at a wave-uniform index is a scalar
// load (no vector registers, not counted with the vector-memory loads).
typedef __attribute__((address_space(4))) const float cfloat;
__device__ __forceinline__ float uniform_load(const float* p, int i) {
  return reinterpret_cast<const cfloat*>(reinterpret_cast<uintptr_t>(p))[i];
}
// Fourth word of a raw buffer descriptor (32-bit data format) and the
// non-temporal cache policy of a buffer load.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kNonTemporal = 2;

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

// P floats held as one vector value: the butterfly's selects between its
// elements then stay selects between registers.
template <int P>
struct FVec {
  typedef float type __attribute__((ext_vector_type(P)));
};

// Lane exchanges of the butterfly below, all VALU (no LDS crossbar):
//  * v_permlane32_swap / v_permlane16_swap exchange the upper half of one
//    register's 64- / 32-lane groups with the lower half of another's; the sum
//    of the two results is, in the lower half of each group, x[l] + x[l ^ o]
//    and, in the upper half, y[l] + y[l ^ o] (o = 32 / 16) - one transposing
//    butterfly step for the pair (x, y) in one swap and one add;
//  * DPP row_ror:8 and quad permutations read lane l ^ 8, l ^ 2, l ^ 1;
//  * DPP row_half_mirror pairs lanes l and 7 - l of an 8-lane group.
// (Lane mappings checked on the device.)
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppRor8 = 0x128, kDppHalfMirror = 0x141, kDppXor2 = 0x4E, kDppXor1 = 0xB1;

template <int O>
__device__ __forceinline__ float lane_xor(float v) {
  if constexpr (O == 8) return dpp<kDppRor8>(v);
  else if constexpr (O == 2) return dpp<kDppXor2>(v);
  else if constexpr (O == 1) return dpp<kDppXor1>(v);
  else return __shfl_xor(v, O, 64);
}

// One step of the transposing butterfly over the lanes of a group, at lane
// distance O with CNT values per lane still to be reduced, then the rest.
template <int O, int CNT, int P>
__device__ __forceinline__ void xstep(typename FVec<P>::type& v, int lane) {
  if constexpr (O >= 1) {
    if constexpr (CNT > 1) {
      constexpr int H = CNT / 2;
      const bool upper = (lane & O) != 0;
#pragma unroll
      for (int i = 0; i < H; ++i) {
        if constexpr (O == 32 || O == 16) {
          const auto r = O == 32
              ? __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]), __float_as_uint(v[i + H]), false, false)
              : __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]), __float_as_uint(v[i + H]), false, false);
          v[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
        } else {
          const float t0 = v[i] + lane_xor<O>(v[i]);
          const float t1 = v[i + H] + lane_xor<O>(v[i + H]);
          v[i] = upper ? t1 : t0;
        }
      }
      xstep<O / 2, H, P>(v, lane);
    } else if constexpr (O == 4) {
      // plain sum over the 8 lanes of a group: mirror pairs, then quads
      float t = v[0] + dpp<kDppHalfMirror>(v[0]);
      t += dpp<kDppXor2>(t);
      v[0] = t + dpp<kDppXor1>(t);
    } else {
      if constexpr (O == 32 || O == 16) {
        const uint32_t u = __float_as_uint(v[0]);
        const auto r = O == 32 ? __builtin_amdgcn_permlane32_swap(u, u, false, false)
                               : __builtin_amdgcn_permlane16_swap(u, u, false, false);
        v[0] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
      } else {
        v[0] += lane_xor<O>(v[0]);
      }
      xstep<O / 2, 1, P>(v, lane);
    }
  }
}

// Transposing butterfly over the LPR lanes of a group.  On return, if
// P <= LPR, lane c of the group holds the total of value c >> (log2 LPR -
// log2 P) in v[0]; otherwise it holds values c*P/LPR .. (c+1)*P/LPR - 1.
template <int P, int LPR>
__device__ __forceinline__ void xreduce(typename FVec<P>::type& v, int lane) {
  xstep<LPR / 2, P, P>(v, lane);
}

constexpr int kBS = 512;  // threads per block

template <int LPR>
struct GemvShape {
  static constexpr int GPW = 64 / LPR;             // lane groups (rows) per wave
  static constexpr int RPI = (kBS / 64) * GPW;     // rows per block iteration
};

// Minimum waves per SIMD the register allocation aims for: 6 where that
// holds without spilling (checked per instantiation: a reload inside the
// main loop would make the wave wait for all of its weight loads), else 4.
template <int MR, int LPR, int UNR, int WT, int EPI>
constexpr int gemv_waves() {
  if (UNR == 4) return MR <= 4 ? 6 : 4;
  if (MR <= (EPI == kEpiFuse ? 1 : 2)) return 6;
  return (LPR == 64 && WT == 0 && EPI == kEpiCloud && MR <= 5) ? 6 : 4;
}

template <int MR, int LPR, int UNR, int WT, int EPI>
__global__ __launch_bounds__(kBS) __attribute__((amdgpu_waves_per_eu(gemv_waves<MR, LPR, UNR, WT, EPI>(), 8)))
void k_gemv(const GemvArgs a) {
  constexpr int GPW = GemvShape<LPR>::GPW, RPI = GemvShape<LPR>::RPI;
  constexpr int EPC = WT == 0 ? 8 : 16;  // weight elements per 16-byte chunk
  constexpr int HW = EPC / 2;            // h words (bf16 pairs) per chunk
  constexpr int P = pow2ceil(MR);
  constexpr int PER = P > LPR ? P / LPR : 1;

  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ uint32_t s_amax[MR];
  __shared__ unsigned long long s_best[MR];
  __shared__ float s_hsc[MR];  // fuse: row factors of int8 hidden-state codes

  const int Kp = a.Kp;
  uint16_t* hs = reinterpret_cast<uint16_t*>(smem);
  int32_t* s_ids = reinterpret_cast<int32_t*>(smem + (size_t)MR * Kp * 2);
  const int tid = threadIdx.x;
  const int n = a.n;
  const int r0 = blockIdx.x * a.rows_per_block;
  const int r1 = min(n, r0 + a.rows_per_block);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int cl = lane % LPR;
  const int grp = wave * GPW + lane / LPR;
  const int nchunk = Kp / EPC;

  // Item stream: item t = (iteration t / passes, pass t % passes); in
  // iteration it the group owns position r0 + it * RPI + grp.
  const int passes = nchunk > 0 ? (nchunk + LPR * UNR - 1) / (LPR * UNR) : 1;
  const int iters = (r1 - r0 + RPI - 1) / RPI;
  const int T = (r1 > r0 && nchunk > 0) ? iters * passes : 0;
  // Position of the group in iteration it, clamped to the block's last
  // position (whose row is then read again but not reported).
  auto pos_of = [&](int it) { return min(r0 + it * RPI + grp, r1 - 1); };

  // After the reduction, reduced value i of this lane is h row own_m[i].
  int own_m[PER];
  bool own[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if constexpr (P > LPR) {
      own_m[i] = cl * PER + i;
      own[i] = own_m[i] < MR;
    } else {
      constexpr int sh = ilog2(LPR) - ilog2(P);
      own_m[i] = cl >> sh;
      own[i] = (cl & ((1 << sh) - 1)) == 0 && own_m[i] < MR;
    }
  }

  // Weight-row access.  With LPR == 64 a wave owns one row: it is read
  // through a buffer descriptor in scalar registers whose size is the row's
  // nchunk chunks, so chunks past the row read as zero with no memory access
  // and chunk u of a pass is an immediate offset.  Smaller groups put
  // several rows in a wave: 64-bit row addresses and per-lane chunk offsets
  // clamped to the row's last chunk (their products are skipped).
  uint32_t coff[LPR == 64 ? 1 : UNR];
  auto set_coff = [&](int p) {
    if constexpr (LPR == 64) {
      coff[0] = (uint32_t)(cl + p * UNR * LPR) * 16u;
    } else {
#pragma unroll
      for (int u = 0; u < UNR; ++u) coff[u] = (uint32_t)min(cl + (p * UNR + u) * LPR, nchunk - 1) * 16u;
    }
  };
  auto row_of = [&](int id) {
    const uint64_t x = reinterpret_cast<uint64_t>(a.w) + (uint64_t)((int64_t)id * a.ldw_bytes);
    if constexpr (LPR == 64) {
      const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
      const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
      void* base = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
      return __builtin_amdgcn_make_buffer_rsrc(base, 0, nchunk * 16, kBufferWord3);
    } else {
      return reinterpret_cast<const gbyte*>(x);
    }
  };
  auto load_chunk = [&](auto row, int u) {
    if constexpr (LPR == 64)
      return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                             row, (int)coff[0], u * LPR * 16, kNonTemporal));
    else
      return __builtin_nontemporal_load(reinterpret_cast<const gu32x4*>(row + coff[u]));
  };

  // Epilogue operands of the values a lane owns in iteration it: the fp8
  // row scale and the bias (cloud), or the payload code and its scale
  // (fuse; 8-bit codes are bytes, 4-bit codes nibbles, one scale per row or
  // per row and block of 2^qshift positions).  Every lane
  // loads them, from index 0 where it has none, so the loads are
  // unconditional and go out with the item's first weight chunk: no load in
  // an epilogue makes the wave wait for the next item's weight loads.
  struct Epi {
    float e0[PER], e1[PER];
  };
  // With LPR == 64 the cloud operands are wave-uniform and are read with
  // scalar loads in the epilogue instead.
  constexpr bool kScalarEpi = EPI == kEpiCloud && LPR == 64;
  auto load_epi = [&](int it, int id, Epi& e) {
    const int j = r0 + it * RPI + grp;
    if constexpr (kScalarEpi) return;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if constexpr (EPI == kEpiCloud) {
        e.e0[i] = WT == 1 ? a.wscale[id] : 1.0f;
        const float* bp = a.bias ? a.bias : a.wscale;  // any valid float array when unused
        const float b = (a.bias || WT == 1) ? bp[(a.bias ? id : 0)] : 0.0f;
        e.e1[i] = a.bias ? b : 0.0f;
      } else {
        const bool ok = own[i] && j < r1;
        const int64_t rq = (int64_t)own_m[i] * a.qstride;
        const uint8_t byte = a.q[ok ? rq + (a.qbits == 8 ? j : (j >> 1)) : 0];
        int code;
        if (a.qbits == 8) {
          code = (int)(int8_t)byte;
        } else {
          const int nib = (j & 1) ? (byte >> 4) : (byte & 15);
          code = nib >= 8 ? nib - 16 : nib;
        }
        e.e0[i] = ok ? (float)code : 0.0f;
        e.e1[i] = a.qscale[ok ? (int64_t)own_m[i] * a.qnb + (a.qshift < 0 ? 0 : (j >> a.qshift)) : 0];
      }
    }
  };

  // The first item's weight loads go out before h is staged, so the staging
  // overlaps them.
  u32x4_t cur[UNR];
  Epi ecur;
#pragma unroll
  for (int i = 0; i < PER; ++i) ecur.e0[i] = ecur.e1[i] = 0.0f;
  if (T > 0) {
    set_coff(0);
    const int id = a.ids[pos_of(0)];
    const auto row = row_of(id);
#pragma unroll
    for (int u = 0; u < UNR; ++u) cur[u] = load_chunk(row, u);
    load_epi(0, id, ecur);
  }

  if (tid < MR) {
    s_amax[tid] = 0u;
    s_best[tid] = 0ull;
  }
  // Stage h[0:MR, 0:K] into LDS, zero padded to Kp, and this block's ids.
  // int8 hidden-state codes are staged as bf16 (exact: at most 8 significant
  // bits) and their row scales applied to the dot products in the epilogue.
  if (EPI == kEpiFuse && a.hq) {
    for (int idx = tid; idx < MR * Kp; idx += kBS) {
      const int m = idx / Kp, k = idx - m * Kp;
      hs[idx] = k < a.K ? (uint16_t)(__float_as_uint((float)a.hq[(int64_t)m * a.ldhq + k]) >> 16)
                        : (uint16_t)0;
    }
    if (tid < MR) s_hsc[tid] = a.hscale[tid];
  } else if ((reinterpret_cast<uintptr_t>(a.h) & 15) == 0 && (a.ldh & 7) == 0 && (a.K & 7) == 0) {
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

  float run_amax[PER];
  unsigned long long run_key[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    run_amax[i] = 0.0f;
    run_key[i] = 0ull;
  }
  float acc[MR];
#pragma unroll
  for (int m = 0; m < MR; ++m) acc[m] = 0.0f;

  // Products of chunk u of the current item; hp0 is this lane's first h
  // element of the item's pass in row 0 of hs.
  auto products = [&](int u, const uint16_t* hp0) {
#pragma unroll
    for (int m = 0; m < MR; ++m) {
      const uint32_t* hp = reinterpret_cast<const uint32_t*>(hp0 + m * Kp + u * LPR * EPC);
      uint32_t hw[HW];
#pragma unroll
      for (int e = 0; e < HW; e += 4) {
        const u32x4_t x = *reinterpret_cast<const u32x4_t*>(hp + e);
        hw[e] = x.x; hw[e + 1] = x.y; hw[e + 2] = x.z; hw[e + 3] = x.w;
      }
      float s = acc[m];
      if constexpr (WT == 0) {
        s = dot2_bf16(cur[u].x, hw[0], s);
        s = dot2_bf16(cur[u].y, hw[1], s);
        s = dot2_bf16(cur[u].z, hw[2], s);
        s = dot2_bf16(cur[u].w, hw[3], s);
      } else {
        const uint32_t w4[4] = {cur[u].x, cur[u].y, cur[u].z, cur[u].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s = dot2_bf16(e4m3x2_to_bf16x2<false>(w4[e]), hw[2 * e], s);
          s = dot2_bf16(e4m3x2_to_bf16x2<true>(w4[e]), hw[2 * e + 1], s);
        }
      }
      acc[m] = s;
    }
  };
  // Reduction and epilogue of iteration it (after its last pass).
  auto finish = [&](int it, const Epi& e) {
    typename FVec<P>::type vals;
#pragma unroll
    for (int i = 0; i < P; ++i) vals[i] = i < MR ? acc[i] : 0.0f;
    xreduce<P, LPR>(vals, lane);
    const int j = r0 + it * RPI + grp;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int m = own_m[i];
      if (!own[i] || j >= r1) continue;
      const float dot = vals[i];
      if constexpr (kScalarEpi) {
        const int id = __builtin_amdgcn_readfirstlane(s_ids[j - r0]);
        const float sc = WT == 1 ? uniform_load(a.wscale, id) : 1.0f;
        const float b = a.bias ? uniform_load(a.bias, id) : 0.0f;
        const float z = dot * sc + b;
        a.z[(int64_t)m * n + j] = z;
        const float y = fminf(fmaxf(z, -a.clip), a.clip);
        run_amax[i] = fmaxf(run_amax[i], fabsf(y));
      } else if constexpr (EPI == kEpiCloud) {
        const float z = dot * e.e0[i] + e.e1[i];
        a.z[(int64_t)m * n + j] = z;
        const float y = fminf(fmaxf(z, -a.clip), a.clip);
        run_amax[i] = fmaxf(run_amax[i], fabsf(y));
      } else {
        const float ze = a.hscale ? dot * s_hsc[m] : dot;
        const float f = __builtin_fmaf(e.e0[i], e.e1[i], ze);
        if (a.f) a.f[(int64_t)m * n + j] = f;
        const unsigned long long key = argmax_key(f, j);
        run_key[i] = key > run_key[i] ? key : run_key[i];
      }
    }
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[m] = 0.0f;
  };

  // Items 0 .. T-2: chunk u is consumed and its registers are refilled at
  // once with chunk u of the next item, so about UNR loads per lane stay in
  // flight through the products and the epilogue.  The last item, which
  // loads nothing, is peeled off so that the loop's loads are unconditional
  // and the compiler's wait counts stay exact.
  int it = 0, pass = 0;
  for (int t = 0; t + 1 < T; ++t) {
    const int npass = pass + 1 == passes ? 0 : pass + 1;
    const int nit = npass == 0 ? it + 1 : it;
    const int nid = s_ids[pos_of(nit) - r0];
    const auto nrow = row_of(nid);
    const uint16_t* hp0 = hs + (cl + pass * UNR * LPR) * EPC;
    const int c0 = cl + pass * UNR * LPR;
    if (passes > 1) set_coff(npass);
    Epi enext = ecur;
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      if (c0 + u * LPR < nchunk) products(u, hp0);
      cur[u] = load_chunk(nrow, u);
      if (u == 0 && npass == 0) load_epi(nit, nid, enext);
    }
    if (pass == passes - 1) finish(it, ecur);
    ecur = enext;
    it = nit;
    pass = npass;
  }
  if (T > 0) {
    const uint16_t* hp0 = hs + (cl + pass * UNR * LPR) * EPC;
    const int c0 = cl + pass * UNR * LPR;
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (c0 + u * LPR < nchunk) products(u, hp0);
    finish(it, ecur);
  }

#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (!own[i]) continue;
    const int m = own_m[i];
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

int gemv_rows_per_iter(int lpr) { return (kBS / 64) * (64 / lpr); }

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
