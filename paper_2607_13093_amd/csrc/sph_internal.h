// Internal declarations shared by the host layer and the kernel files.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <vector>
#include <stddef.h>
#include <stdint.h>

namespace sph {

// While a trace region is open on this thread (sph_trace_start), launches
// carry the region's events on the dispatch itself: the start event on the
// first kernel, the stop event on every kernel (the last one wins), so the
// recorded interval is kernel execution only.
struct TraceEvents {
  hipEvent_t start, stop;
  bool launched;
};
extern thread_local TraceEvents* t_trace_events;

template <class K, class... Args>
inline void launch_kernel(K kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t s,
                          Args... args) {
  TraceEvents* te = t_trace_events;
  if (te) {
    hipExtLaunchKernelGGL(kernel, grid, block, lds, s, te->launched ? nullptr : te->start,
                          te->stop, 0u, args...);
    te->launched = true;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
  }
}

// Per-block / per-tile partial results are stored [M][kMaxBlocks]; no
// projection launch produces more column partials than this.
constexpr int kMaxBlocks = 2048;
// Largest LDS footprint the skinny kernels give to the staged rows of h.
constexpr int kGemvLdsBytes = 60 * 1024;
// Largest row count handled by one skinny launch.
constexpr int kGemvMaxRows = 8;
// Largest contiguous share of subset positions one skinny block stages.
constexpr int kGemvMaxIdsPerBlock = 2048;

// Arguments of the skinny (VALU) gathered projection.  One launch covers up
// to kGemvMaxRows rows of h and every subset id.
struct GemvArgs {
  const uint16_t* h;      // bf16 [rows, ldh]
  int64_t ldh;
  int K;                  // reduction length (d_cloud or d_end)
  int Kp;                 // K rounded up to the weight chunk (8 bf16 / 16 fp8)
  const uint8_t* w;       // weight rows, vocab-major
  int64_t ldw_bytes;      // row stride of w in bytes
  const float* wscale;    // fp32 [V] for fp8 weights, else null
  const int32_t* ids;     // subset ids [n]
  int n;
  int nblk;               // partial slots per row the consumer reads (<= kMaxBlocks);
                          // the launch may use fewer blocks and zero-fills the rest
  int rows_per_block;     // set by the launcher: contiguous positions per block
  // cloud epilogue
  const float* bias;      // fp32 [V] or null
  float clip;
  float* z;               // fp32 [rows, n]
  float* amax_part;       // fp32 [rows, kMaxBlocks]
  // fuse epilogue: the payload in format (qbits, block of 2^qshift positions
  // or one per row when qshift < 0)
  const uint8_t* q;       // codes, rows of qstride bytes
  int64_t qstride;
  const float* qscale;    // fp32 [rows, qnb]
  int qbits, qshift, qnb;
  float* f;               // fp32 [rows, n] or null
  uint64_t* best_part;    // argmax keys [rows, kMaxBlocks]
  // fuse only: int8 hidden-state codes instead of bf16 h (then h is unused)
  // and their row scales, which multiply the row's dot products
  const int8_t* hq;       // [rows, ldhq] or null
  int64_t ldhq;
  const float* hscale;    // fp32 [rows] or null
};

// Arguments of the dense (MFMA) gathered projection: C = h[M, K] * W[S]^T.
struct MfmaArgs {
  const uint16_t* h;      // bf16 [M, ldh], 16-byte aligned rows
  int64_t ldh;
  int M;
  int K;                  // multiple of 8 (bf16 weights) or 16 (fp8 weights)
  const uint8_t* w;       // weight rows, vocab-major, 16-byte aligned
  int64_t ldw_bytes;
  int64_t w_rows;         // rows of w the ids address (the vocabulary); 0 if unknown
  const float* wscale;    // fp32 [V] for fp8 weights, else null
  const int32_t* ids;     // subset ids [n]
  int n;
  int m_tiles, n_tiles;   // set by the launcher
  // cloud epilogue
  const float* bias;
  float clip;
  float* z;               // fp32 [M, n]
  float* amax_part;       // fp32 [M, kMaxBlocks], slot = n-tile
  // fuse epilogue: the payload in format (qbits, block of 2^qshift >= 256
  // positions or one per row when qshift < 0)
  const uint8_t* q;       // codes, rows of qstride bytes
  int64_t qstride;
  const float* qscale;    // fp32 [M, qnb]
  int qbits, qshift, qnb;
  float* f;               // fp32 [M, n] or null
  uint64_t* best_part;    // argmax keys [M, kMaxBlocks], slot = n-tile
  const float* hscale;    // fuse only: fp32 [M] factors of the dot products, or null
  // cloud with the payload quantised in the epilogue (scale blocks of one
  // 256-position tile): codes rows of qout_stride bytes, scales [M, qout_nb];
  // z is then written only if non-null
  uint8_t* qout;
  int64_t qout_stride;
  float* qout_scale;
  int qout_bits, qout_nb;
};

constexpr int kMfmaBN = 256;  // subset positions per MFMA tile

enum Epilogue { kEpiCloud = 0, kEpiFuse = 1, kEpiCloudQ = 2 };

// Launchers (return the HIP launch status).
hipError_t launch_gemv(int epi, int wtype, int rows, const GemvArgs& a, hipStream_t s);
int gemv_rows_per_iter(int lpr);
int gemv_lpr(int K, int wtype);

hipError_t launch_mfma(int epi, int wtype, const MfmaArgs& a, hipStream_t s);
// true where the cloud projection can quantise blocks of 256 positions in its epilogue
bool mfma_quantises_in_epilogue(int M, int K);
int mfma_n_tiles(int n);

// Clip + quantise z [M, n] to b-bit codes (bits 8 or 4; 4-bit codes two per
// byte, low nibble first) with one scale per row (qshift < 0: from the
// projection's per-block maxima amax_part) or per row and block of 2^qshift
// positions (8 <= qshift <= 12).  q rows are qstride bytes, scale rows qnb.
hipError_t launch_quantize(const float* z, const float* amax_part, int nblk, int M, int n,
                           float clip, int bits, int qshift, uint8_t* q, int64_t qstride,
                           float* scale, int qnb, hipStream_t s);

// best/nblk: the endpoint projection's per-tile argmax keys of each row
// (row stride kMaxBlocks), whose maximum gives the row's largest logit.
hipError_t launch_sample(const float* f, int M, int n, const unsigned long long* best, int nblk,
                         const int32_t* ids, int R, float temperature, float top_p, uint64_t seed,
                         int32_t* tokens, hipStream_t s);
hipError_t launch_accept(const int32_t* tokens, const int32_t* drafts, int n_sessions, int R,
                         int32_t* accept, hipStream_t s);

hipError_t launch_final_greedy(const uint64_t* best_part, int nblk, const int32_t* ids, int n,
                               int n_sessions, int R, const int32_t* drafts,
                               int32_t* tokens, int32_t* accept, hipStream_t s);

// Hidden-state codes (hidden.hip): per-row int8 codes and scales of bf16
// rows h [M, ldh] (d columns), and the widening of codes [M, ldhq] (K
// columns) into bf16 operands out [M, Kp] (Kp a multiple of 8, pad zero).
hipError_t launch_hidden_quantize(const uint16_t* h, int64_t ldh, int M, int d, int8_t* q,
                                  int64_t ldq, float* scale, hipStream_t s);
hipError_t launch_widen_codes(const int8_t* hq, int64_t ldhq, int M, int K, int Kp,
                              uint16_t* out, hipStream_t s);

// AES-GCM of payload rows (gcm.hip).  A key's device image holds the T0
// table (1 KB), the S-box (256 B), the round keys (at kGcmRkOffset), the
// powers H^0 .. H^kGcmMaxPow of the hash key (16 B each, at kGcmPowOffset)
// and, at kGcmTabOffset, the product by G = H^kGcmStride as 32 nibble
// tables: entry [p][v] (16 B) is G times the block whose nibble p (from the
// most significant end) is v and whose other bits are zero.
constexpr int kGcmMaxPow = 16384;  // AAD + ciphertext + length blocks of one message
constexpr int kGcmRkOffset = 1280;
constexpr int kGcmPowOffset = 1536;
constexpr int kGcmStride = 256;    // blocks between the terms one thread chains
constexpr int kGcmMaxChain = 16;   // blocks one thread chains at most
constexpr size_t kGcmTabOffset = (size_t)kGcmPowOffset + (size_t)(kGcmMaxPow + 1) * 16;
constexpr size_t kGcmImageBytes = kGcmTabOffset + 32 * 16 * 16;
bool gcm_key_setup(const uint8_t* key, int key_bytes, std::vector<uint8_t>& dev_image, int& nr);
// A message row is the concatenation of up to kGcmMaxSegs segments: bytes
// [end[k-1], end[k]) of row r come from in[k] + r * ld_in[k] and go to
// out[k] + r * ld_out[k] (end[-1] = 0; empty segments allowed).  Passed to
// the kernels by value.
constexpr int kGcmMaxSegs = 4;
struct GcmSegs {
  const uint8_t* in[kGcmMaxSegs];
  uint8_t* out[kGcmMaxSegs];
  int64_t ld_in[kGcmMaxSegs];
  int64_t ld_out[kGcmMaxSegs];
  int64_t end[kGcmMaxSegs];
  int nseg;
};
constexpr int kGcmMaxAad = 1024;  // bytes of associated data per message
// Blocks each thread chains for a batch of rows messages of n data blocks:
// 1 while the batch has few blocks (parallelism first), up to kGcmMaxChain
// for large batches.
inline int gcm_chain(int64_t rows, int64_t n) {
  const int64_t k = (rows * n + 32767) / 32768;
  return (int)(k < 1 ? 1 : (k > kGcmMaxChain ? kGcmMaxChain : k));
}
// Workgroups (of kGcmStride threads) per message of n data blocks and na
// AAD blocks.  The last na + 2 threads of workgroup *extra_part take the
// AAD blocks, the length block and E_K(J0): the last data workgroup, unless
// threads chain single blocks (a latency-bound batch) and it has fewer than
// na + 2 threads without a block; then one more workgroup.  (Adding a
// workgroup per row to a large batch would double its grid.)
inline int gcm_parts(int64_t n, int64_t na, int chain, int* extra_part = nullptr) {
  const int64_t per = (int64_t)kGcmStride * chain;
  const int64_t nd = (n + per - 1) / per;
  const int64_t in_last = nd > 0 ? n - (nd - 1) * per : kGcmStride;
  const int64_t idle = in_last < kGcmStride ? kGcmStride - in_last : 0;
  const int64_t xp = nd > 0 && (chain > 1 || idle >= na + 2) ? nd - 1 : nd;
  if (extra_part) *extra_part = (int)xp;
  return (int)(xp + 1);
}
// rows <= 65535 messages of L = segs.end[nseg-1] bytes with la <= kGcmMaxAad
// bytes of AAD; partial: rows * gcm_parts(n, ceil(la/16), gcm_chain(rows, n))
// * 16 bytes with n = ceil(L/16)
hipError_t launch_gcm(bool open, const uint8_t* key_dev, int nr, const GcmSegs& segs, int rows,
                      const uint8_t* iv, const uint8_t* aad, int64_t ld_aad, int la, uint8_t* tag,
                      int32_t* ok, uint32_t* partial, hipStream_t s);

// Measurement kernels (probe.hip).
hipError_t launch_probe_read(const void* buf, int64_t bytes, float* sink, hipStream_t s);
hipError_t launch_probe_mfma(int iters, float* sink, hipStream_t s);
double probe_mfma_flops(int64_t iters);

}  // namespace sph
