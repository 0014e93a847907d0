// C-ABI host layer: argument validation, subset plans, workspace layout and
// dispatch of the kernels on the caller's stream.  Nothing here touches
// device data; every check happens before the first launch.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <vector>

#include "sph.h"
#include "sph_probe.h"
#include "sph_internal.h"

struct sph_subset_s {
  int32_t* d_ids;   // device int32 [n], strictly ascending
  int64_t n;
  int64_t vocab;
  int device;
};

struct sph_gcm_key_s {
  uint8_t* d_image;  // T0 | S-box | round keys | powers of H (device)
  int nr;            // AES rounds: 10 (128-bit key) or 14 (256-bit key)
};

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return SPH_OK;
}

// Set by a failing debug synchronisation (see traced) to name the kernel the
// error surfaced after; consumed by the next hip_fail on this thread.
thread_local std::string t_sync_note;

int hip_fail(hipError_t e, const char* what) {
  if (!t_sync_note.empty()) {
    const std::string note = t_sync_note;
    t_sync_note.clear();
    return fail(SPH_E_DEVICE, "%s (%s): %s", what, note.c_str(), hipGetErrorString(e));
  }
  return fail(SPH_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Debug mode: every launch region is followed by a synchronisation of its
// stream and an error check, so a failing kernel is reported by the call
// that launched it.  Off by default; SPH_DEBUG_SYNC=1 in the environment
// turns it on at the first call, sph_debug_sync() at any time.
std::atomic<int> g_debug_sync{-1};

bool debug_sync_on() {
  int v = g_debug_sync.load(std::memory_order_acquire);
  if (v < 0) {
    const char* env = std::getenv("SPH_DEBUG_SYNC");
    const int want = (env && env[0] && env[0] != '0') ? 1 : 0;
    int expected = -1;
    g_debug_sync.compare_exchange_strong(expected, want, std::memory_order_acq_rel);
    v = g_debug_sync.load(std::memory_order_acquire);
  }
  return v > 0;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

constexpr int64_t kMaxIds = 0x7FFFFFFF;

}  // namespace

namespace sph {
thread_local TraceEvents* t_trace_events = nullptr;
}  // namespace sph

namespace {

// ---- kernel tracing: events attached to the dispatches of a region --------
struct TraceSlot {
  const char* name;
  hipEvent_t start, stop;
  bool used;
};
// The trace is process-wide: g_trace and g_trace_used are guarded by
// g_trace_mu; g_tracing is read without the lock (acquire) on every launch
// and written under it (release), so an untraced launch costs one load.
std::mutex g_trace_mu;
std::vector<TraceSlot> g_trace;
size_t g_trace_used = 0;
std::atomic<bool> g_tracing{false};

void trace_free_locked() {
  for (auto& t : g_trace) {
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  g_trace.clear();
  g_trace_used = 0;
  g_tracing.store(false, std::memory_order_release);
}

// Launch `body` (returning hipError_t); while tracing, its kernels record the
// slot's events on their dispatches (see launch_kernel).  In debug mode the
// stream is synchronised afterwards (unless it is being captured into a
// graph) and an execution error is returned as the region's error.
template <class F>
hipError_t traced(const char* name, hipStream_t s, F&& body) {
  long slot = -1;
  sph::TraceEvents ev{nullptr, nullptr, false};
  if (g_tracing.load(std::memory_order_acquire)) {
    std::lock_guard<std::mutex> lk(g_trace_mu);
    if (g_tracing.load(std::memory_order_relaxed) && g_trace_used < g_trace.size()) {
      slot = (long)g_trace_used++;
      g_trace[(size_t)slot].name = name;
      g_trace[(size_t)slot].used = false;
      ev.start = g_trace[(size_t)slot].start;
      ev.stop = g_trace[(size_t)slot].stop;
    }
  }
  if (slot >= 0) sph::t_trace_events = &ev;
  hipError_t e = body();
  sph::t_trace_events = nullptr;
  if (slot >= 0) {
    std::lock_guard<std::mutex> lk(g_trace_mu);
    if ((size_t)slot < g_trace.size()) g_trace[(size_t)slot].used = ev.launched;
  }
  if (e == hipSuccess && debug_sync_on()) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    hipError_t ce = hipStreamIsCapturing(s, &cs);
    if (ce == hipSuccess && cs == hipStreamCaptureStatusNone) {
      e = hipStreamSynchronize(s);
      if (e == hipSuccess) e = hipGetLastError();
      if (e != hipSuccess) t_sync_note = std::string("debug sync after ") + name;
    } else if (ce != hipSuccess) {
      e = ce;
    }
  }
  return e;
}

// log2(block) for a payload block of 256 ... 4096 positions (a power of two),
// -1 for block 0 (one scale per row), -2 for anything else.
int block_shift(int64_t block) {
  if (block == 0) return -1;
  for (int sh = 8; sh <= 12; ++sh)
    if (block == (int64_t(1) << sh)) return sh;
  return -2;
}

int make_plan(const int32_t* host_ids, int64_t n, int64_t vocab, hipStream_t stream,
              sph_subset* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int32_t* d = nullptr;
  e = hipMalloc(&d, (size_t)n * sizeof(int32_t));
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(subset)");
  e = hipMemcpyAsync(d, host_ids, (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    (void)hipFree(d);
    return hip_fail(e, "copying subset ids");
  }
  *out = new sph_subset_s{d, n, vocab, dev};
  return ok();
}

// Cloud workspace: [fp32 z : M x n][fp32 row-max partials : M x kMaxBlocks]
size_t cloud_ws(int64_t M, int64_t n) {
  if (M <= 0) return 0;
  return align256((size_t)M * n * 4) + align256((size_t)M * sph::kMaxBlocks * 4);
}

// Fuse workspace: [argmax keys : M x kMaxBlocks][sample: fp32 f : M x n]
size_t fuse_ws(int64_t M, int64_t n, int mode) {
  if (M <= 0) return 0;
  size_t b = align256((size_t)M * sph::kMaxBlocks * 8);
  if (mode == SPH_SAMPLE) b += align256((size_t)M * n * 4);
  return b;
}

// int8 hidden-state codes of more rows than the skinny projection takes are
// widened to bf16 operands [M, round_up(d_end, 8)] after the fuse workspace.
size_t widen_ws(int64_t M, int64_t d_end) {
  if (M <= sph::kGemvMaxRows || d_end <= 0) return 0;
  return align256((size_t)M * (size_t)((d_end + 7) / 8 * 8) * 2);
}

// ---- allocation-free cloud call -------------------------------------------
// A file-scope device array stands in for the caller's workspace.  Each GPU
// holds its own copy at its own address; the host never passes `scratch`
// itself to a kernel (its host-side name is not a device address) but the
// address hipGetSymbolAddress returns, looked up once per device with that
// device current and kept in g_scratch_addr.
constexpr size_t kScratchBytes = size_t(SPH_NOALLOC_SCRATCH_BYTES);
__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of this device's scratch (the current device), or an error.
int scratch_address(const char* fn, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(SPH_E_UNSUPPORTED, "%s: device %d beyond the %d the library tracks", fn, dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(SPH_E_DEVICE, "%s: no device address for the scratch array", fn);
    g_scratch_addr[dev] = ptr;
  }
  *out = g_scratch_addr[dev];
  return SPH_OK;
}

}  // namespace

extern "C" {

int sph_abi_version(void) { return SPH_ABI_VERSION; }

int sph_debug_sync(int enable) {
  const int prev = debug_sync_on() ? 1 : 0;
  if (enable >= 0) g_debug_sync.store(enable ? 1 : 0, std::memory_order_release);
  return prev;
}

const char* sph_last_error(void) { return g_err.c_str(); }

int sph_subset_create(const int32_t* host_ids, int64_t n, int64_t vocab, void* stream,
                      sph_subset* out) {
  if (!out) return fail(SPH_E_INVALID_ARG, "sph_subset_create: out is NULL");
  *out = nullptr;
  if (!host_ids) return fail(SPH_E_INVALID_ARG, "sph_subset_create: host_ids is NULL");
  if (vocab < 1 || vocab > kMaxIds)
    return fail(SPH_E_INVALID_ARG, "sph_subset_create: vocab %lld out of range", (long long)vocab);
  if (n < 1 || n > vocab)
    return fail(SPH_E_SUBSET, "sph_subset_create: size %lld not in [1, vocab=%lld]", (long long)n,
                (long long)vocab);
  for (int64_t i = 0; i < n; ++i) {
    const int64_t id = host_ids[i];
    if (id < 0 || id >= vocab)
      return fail(SPH_E_SUBSET, "sph_subset_create: id %lld at %lld outside [0, %lld)",
                  (long long)id, (long long)i, (long long)vocab);
    if (i > 0 && id <= host_ids[i - 1])
      return fail(SPH_E_SUBSET, "sph_subset_create: ids not strictly ascending at %lld (%d after %d)",
                  (long long)i, (int)id, (int)host_ids[i - 1]);
  }
  return make_plan(host_ids, n, vocab, (hipStream_t)stream, out);
}

int sph_subset_create_full(int64_t vocab, void* stream, sph_subset* out) {
  if (!out) return fail(SPH_E_INVALID_ARG, "sph_subset_create_full: out is NULL");
  *out = nullptr;
  if (vocab < 1 || vocab > kMaxIds)
    return fail(SPH_E_INVALID_ARG, "sph_subset_create_full: vocab %lld out of range",
                (long long)vocab);
  std::vector<int32_t> ids((size_t)vocab);
  for (int64_t i = 0; i < vocab; ++i) ids[(size_t)i] = (int32_t)i;
  return make_plan(ids.data(), vocab, vocab, (hipStream_t)stream, out);
}

int sph_subset_size(sph_subset subset, int64_t* n, int64_t* vocab) {
  if (!subset) return fail(SPH_E_INVALID_ARG, "sph_subset_size: subset is NULL");
  if (n) *n = subset->n;
  if (vocab) *vocab = subset->vocab;
  return ok();
}

int sph_subset_device_ids(sph_subset subset, const int32_t** ids) {
  if (!subset || !ids) return fail(SPH_E_INVALID_ARG, "sph_subset_device_ids: NULL argument");
  *ids = subset->d_ids;
  return ok();
}

void sph_subset_destroy(sph_subset subset) {
  if (!subset) return;
  (void)hipFree(subset->d_ids);
  delete subset;
}

size_t sph_cloud_partial_workspace(int64_t M, sph_subset subset) {
  if (!subset || M < 0) return 0;
  return cloud_ws(M, subset->n);
}

size_t sph_fuse_verify_workspace(int64_t M, sph_subset subset, int mode) {
  if (!subset || M < 0) return 0;
  return fuse_ws(M, subset->n, mode);
}

size_t sph_fuse_verify_hq_workspace(int64_t M, int64_t d_end, sph_subset subset, int mode) {
  if (!subset || M < 0 || d_end < 0) return 0;
  return fuse_ws(M, subset->n, mode) + widen_ws(M, d_end);
}

int sph_hidden_quantize(const void* h, int64_t ldh, int64_t M, int64_t d, int8_t* q_out,
                        int64_t ldq, float* scale_out, void* stream) {
  const char* fn = "sph_hidden_quantize";
  if (M < 0 || M > (1 << 24)) return fail(SPH_E_INVALID_ARG, "%s: M=%lld out of range", fn, (long long)M);
  if (d < 0 || d > (1 << 20)) return fail(SPH_E_INVALID_ARG, "%s: d=%lld out of range", fn, (long long)d);
  if (ldh < d || ldq < d)
    return fail(SPH_E_INVALID_ARG, "%s: row strides (ldh=%lld, ldq=%lld) below d=%lld", fn,
                (long long)ldh, (long long)ldq, (long long)d);
  if (M == 0) return ok();
  if (!scale_out || (d > 0 && (!h || !q_out)))
    return fail(SPH_E_INVALID_ARG, "%s: h/q_out/scale_out is NULL", fn);
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = traced("hidden_quantize", s, [&] {
    return sph::launch_hidden_quantize(static_cast<const uint16_t*>(h), ldh, (int)M, (int)d, q_out,
                                       ldq, scale_out, s);
  });
  if (e != hipSuccess) return hip_fail(e, "hidden-state quantiser launch");
  return ok();
}

int64_t sph_payload_code_bytes(int64_t n_sub, int bits) {
  if (n_sub < 0 || (bits != 8 && bits != 4)) return -1;
  return (n_sub * bits + 7) / 8;
}

int64_t sph_payload_scale_count(int64_t n_sub, int64_t block) {
  if (n_sub < 0 || block_shift(block) == -2) return -1;
  return block == 0 ? 1 : std::max<int64_t>(1, (n_sub + block - 1) / block);
}

int sph_cloud_partial(const void* h_cloud, int64_t ldh, int64_t M, int64_t d_cloud,
                      const void* w_cloud, int64_t ldw, int wtype, const float* w_row_scale,
                      const float* bias, sph_subset subset, float clip_c, int8_t* q_out,
                      float* scale_out, float* z_out, void* workspace, size_t ws_bytes,
                      void* stream) {
  return sph_cloud_partial_fmt(h_cloud, ldh, M, d_cloud, w_cloud, ldw, wtype, w_row_scale, bias,
                               subset, clip_c, 8, 0, q_out, scale_out, z_out, workspace, ws_bytes,
                               stream);
}

int sph_cloud_partial_fmt(const void* h_cloud, int64_t ldh, int64_t M, int64_t d_cloud,
                          const void* w_cloud, int64_t ldw, int wtype, const float* w_row_scale,
                          const float* bias, sph_subset subset, float clip_c, int bits,
                          int64_t block, void* q_out, float* scale_out, float* z_out,
                          void* workspace, size_t ws_bytes, void* stream) {
  const char* fn = "sph_cloud_partial";
  if (bits != 8 && bits != 4) return fail(SPH_E_INVALID_ARG, "%s: bits=%d not 4 or 8", fn, bits);
  const int qshift = block_shift(block);
  if (qshift == -2)
    return fail(SPH_E_INVALID_ARG, "%s: block=%lld not 0 or a power of two in [256, 4096]", fn,
                (long long)block);
  if (M < 0 || M > (1 << 24)) return fail(SPH_E_INVALID_ARG, "%s: M=%lld out of range", fn, (long long)M);
  if (d_cloud < 0 || d_cloud > (1 << 20))
    return fail(SPH_E_INVALID_ARG, "%s: d_cloud=%lld out of range", fn, (long long)d_cloud);
  if (wtype != SPH_W_BF16 && wtype != SPH_W_FP8_E4M3)
    return fail(SPH_E_INVALID_ARG, "%s: unknown weight type %d", fn, wtype);
  if (wtype == SPH_W_FP8_E4M3 && !w_row_scale)
    return fail(SPH_E_INVALID_ARG, "%s: fp8 weights need w_row_scale", fn);
  if (wtype == SPH_W_BF16 && w_row_scale)
    return fail(SPH_E_INVALID_ARG, "%s: w_row_scale is only for fp8 weights", fn);
  if (!(clip_c > 0.0f) || !std::isfinite(clip_c))
    return fail(SPH_E_INVALID_ARG, "%s: clip_c must be positive and finite", fn);
  if (ldh < d_cloud || ldw < d_cloud)
    return fail(SPH_E_INVALID_ARG, "%s: row strides (ldh=%lld, ldw=%lld) below d_cloud=%lld", fn,
                (long long)ldh, (long long)ldw, (long long)d_cloud);
  if (!subset) return fail(SPH_E_INVALID_ARG, "%s: subset is NULL", fn);
  if (M == 0) return ok();
  if (!h_cloud && d_cloud > 0) return fail(SPH_E_INVALID_ARG, "%s: h_cloud is NULL", fn);
  if (!w_cloud) return fail(SPH_E_INVALID_ARG, "%s: w_cloud is NULL", fn);
  if (!q_out || !scale_out) return fail(SPH_E_INVALID_ARG, "%s: q_out/scale_out is NULL", fn);
  const int64_t n = subset->n;
  const size_t need = cloud_ws(M, n);
  if (!workspace || ws_bytes < need)
    return fail(SPH_E_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                workspace ? ws_bytes : (size_t)0);
  const int wbytes = wtype == SPH_W_BF16 ? 2 : 1;
  const int epc = wtype == SPH_W_BF16 ? 8 : 16;
  const int64_t Kp = round_up(d_cloud, epc);
  if ((reinterpret_cast<uintptr_t>(w_cloud) & 15) != 0 || (ldw * wbytes) % 16 != 0 || d_cloud % epc != 0)
    return fail(SPH_E_UNSUPPORTED,
                "%s: weight rows must be 16-byte aligned and d_cloud a multiple of %d", fn, epc);
  if (n > (int64_t)sph::kMaxBlocks * sph::kGemvMaxIdsPerBlock)
    return fail(SPH_E_UNSUPPORTED, "%s: subset of %lld ids is too large", fn, (long long)n);

  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float* z = z_out ? z_out : reinterpret_cast<float*>(ws);
  float* amax = reinterpret_cast<float*>(ws + align256((size_t)M * n * 4));

  // Dense path: more rows than one skinny launch covers, 16-byte aligned h rows.
  const bool h_vec = (reinterpret_cast<uintptr_t>(h_cloud) & 15) == 0 && ldh % 8 == 0;
  const int64_t qstride = sph_payload_code_bytes(n, bits);
  const int qnb = (int)sph_payload_scale_count(n, block);
  int nblk;
  if (M > sph::kGemvMaxRows && h_vec && sph::mfma_n_tiles((int)n) <= sph::kMaxBlocks &&
      block == sph::kMfmaBN && sph::mfma_quantises_in_epilogue((int)M, (int)d_cloud)) {
    // a scale block is one 256-position tile: the projection's epilogue
    // quantises from its accumulators, z is written only on request
    sph::MfmaArgs a{};
    a.h = static_cast<const uint16_t*>(h_cloud);
    a.ldh = ldh;
    a.M = (int)M;
    a.K = (int)d_cloud;
    a.w = static_cast<const uint8_t*>(w_cloud);
    a.ldw_bytes = ldw * wbytes;
    a.w_rows = subset->vocab;
    a.wscale = w_row_scale;
    a.ids = subset->d_ids;
    a.n = (int)n;
    a.bias = bias;
    a.clip = clip_c;
    a.z = z_out;
    a.qout = static_cast<uint8_t*>(q_out);
    a.qout_stride = qstride;
    a.qout_scale = scale_out;
    a.qout_bits = bits;
    a.qout_nb = qnb;
    hipError_t e = traced("cloud_mfma", s, [&] { return sph::launch_mfma(sph::kEpiCloudQ, wtype, a, s); });
    if (e != hipSuccess) return hip_fail(e, "cloud projection launch");
    return ok();
  }
  if (M > sph::kGemvMaxRows && h_vec && sph::mfma_n_tiles((int)n) <= sph::kMaxBlocks) {
    sph::MfmaArgs a{};
    a.h = static_cast<const uint16_t*>(h_cloud);
    a.ldh = ldh;
    a.M = (int)M;
    a.K = (int)d_cloud;
    a.w = static_cast<const uint8_t*>(w_cloud);
    a.ldw_bytes = ldw * wbytes;
    a.w_rows = subset->vocab;
    a.wscale = w_row_scale;
    a.ids = subset->d_ids;
    a.n = (int)n;
    a.bias = bias;
    a.clip = clip_c;
    a.z = z;
    a.amax_part = amax;
    hipError_t e = traced("cloud_mfma", s, [&] { return sph::launch_mfma(sph::kEpiCloud, wtype, a, s); });
    if (e != hipSuccess) return hip_fail(e, "cloud projection launch");
    nblk = sph::mfma_n_tiles((int)n);
  } else {
    int mr = sph::kGemvMaxRows;
    if (Kp > 0) mr = (int)std::min<int64_t>(mr, sph::kGemvLdsBytes / (Kp * 2));
    if (mr < 1) return fail(SPH_E_UNSUPPORTED, "%s: d_cloud=%lld too large", fn, (long long)d_cloud);
    const int lpr = sph::gemv_lpr((int)d_cloud, wtype);
    const int rpi = sph::gemv_rows_per_iter(lpr);
    nblk = (int)std::min<int64_t>((n + rpi - 1) / rpi, sph::kMaxBlocks);
    for (int64_t m0 = 0; m0 < M; m0 += mr) {
      const int rows = (int)std::min<int64_t>(mr, M - m0);
      sph::GemvArgs a{};
      a.h = static_cast<const uint16_t*>(h_cloud) + m0 * ldh;
      a.ldh = ldh;
      a.K = (int)d_cloud;
      a.Kp = (int)Kp;
      a.w = static_cast<const uint8_t*>(w_cloud);
      a.ldw_bytes = ldw * wbytes;
      a.wscale = w_row_scale;
      a.ids = subset->d_ids;
      a.n = (int)n;
      a.nblk = nblk;
      a.bias = bias;
      a.clip = clip_c;
      a.z = z + m0 * n;
      a.amax_part = amax + m0 * sph::kMaxBlocks;
      hipError_t e = traced("cloud_gemv", s, [&] { return sph::launch_gemv(sph::kEpiCloud, wtype, rows, a, s); });
      if (e != hipSuccess) return hip_fail(e, "cloud projection launch");
    }
  }
  hipError_t e = traced("cloud_quantize", s, [&] {
    return sph::launch_quantize(z, amax, nblk, (int)M, (int)n, clip_c, bits, qshift,
                                static_cast<uint8_t*>(q_out), qstride, scale_out, qnb, s);
  });
  if (e != hipSuccess) return hip_fail(e, "quantiser launch");
  return ok();
}

int sph_cloud_partial_noalloc(const void* h_cloud, int64_t ldh, int64_t M, int64_t d_cloud,
                              const void* w_cloud, int64_t ldw, int wtype,
                              const float* w_row_scale, const float* bias, sph_subset subset,
                              float clip_c, int bits, int64_t block, void* q_out,
                              float* scale_out, float* z_out, void* stream) {
  const char* fn = "sph_cloud_partial_noalloc";
  if (!subset) return fail(SPH_E_INVALID_ARG, "%s: subset is NULL", fn);
  if (M < 0) return fail(SPH_E_INVALID_ARG, "%s: M=%lld out of range", fn, (long long)M);
  const size_t need = cloud_ws(M, subset->n);
  if (need > kScratchBytes)
    return fail(SPH_E_WORKSPACE,
                "%s: %lld rows x %lld ids need %zu bytes of scratch; the static scratch holds "
                "%zu bytes (use sph_cloud_partial_fmt with a workspace)",
                fn, (long long)M, (long long)subset->n, need, kScratchBytes);
  void* ws = nullptr;
  const int rc = scratch_address(fn, &ws);
  if (rc != SPH_OK) return rc;
  return sph_cloud_partial_fmt(h_cloud, ldh, M, d_cloud, w_cloud, ldw, wtype, w_row_scale, bias,
                               subset, clip_c, bits, block, q_out, scale_out, z_out, ws,
                               kScratchBytes, stream);
}

int sph_fuse_verify(const int8_t* q, const float* scale, const void* h_end, int64_t ldh,
                    int64_t d_end, const void* w_end, int64_t ldw, sph_subset subset,
                    int64_t n_sessions, int64_t rows_per_session, const int32_t* drafts, int mode,
                    float temperature, float top_p, uint64_t seed, int32_t* tokens_out,
                    int32_t* accept_len_out, float* fused_out, void* workspace, size_t ws_bytes,
                    void* stream) {
  return sph_fuse_verify_fmt(q, scale, 8, 0, h_end, ldh, d_end, w_end, ldw, subset, n_sessions,
                             rows_per_session, drafts, mode, temperature, top_p, seed, tokens_out,
                             accept_len_out, fused_out, workspace, ws_bytes, stream);
}

namespace {

// The endpoint call, with the endpoint's hidden state either as bf16 rows
// (h_end, ldh) or as int8 codes with row scales (hq, ldh, h_scale).
int fuse_verify_impl(const char* fn, bool codes, const void* q, const float* scale, int bits,
                     int64_t block, const void* h_end, const int8_t* hq, const float* h_scale,
                     int64_t ldh, int64_t d_end, const void* w_end, int64_t ldw,
                     sph_subset subset, int64_t n_sessions, int64_t rows_per_session,
                     const int32_t* drafts, int mode, float temperature, float top_p,
                     uint64_t seed, int32_t* tokens_out, int32_t* accept_len_out,
                     float* fused_out, void* workspace, size_t ws_bytes, void* stream) {
  if (bits != 8 && bits != 4) return fail(SPH_E_INVALID_ARG, "%s: bits=%d not 4 or 8", fn, bits);
  const int qshift = block_shift(block);
  if (qshift == -2)
    return fail(SPH_E_INVALID_ARG, "%s: block=%lld not 0 or a power of two in [256, 4096]", fn,
                (long long)block);
  if (n_sessions < 0 || rows_per_session < 1 || rows_per_session > 1024)
    return fail(SPH_E_INVALID_ARG, "%s: n_sessions=%lld / rows_per_session=%lld out of range", fn,
                (long long)n_sessions, (long long)rows_per_session);
  const int64_t M = n_sessions * rows_per_session;
  if (M > (1 << 24)) return fail(SPH_E_INVALID_ARG, "%s: M=%lld too large", fn, (long long)M);
  if (d_end < 0 || d_end > (1 << 20))
    return fail(SPH_E_INVALID_ARG, "%s: d_end=%lld out of range", fn, (long long)d_end);
  if (mode != SPH_GREEDY && mode != SPH_SAMPLE)
    return fail(SPH_E_INVALID_ARG, "%s: unknown mode %d", fn, mode);
  if (mode == SPH_SAMPLE) {
    if (!(temperature > 0.0f) || !std::isfinite(temperature))
      return fail(SPH_E_INVALID_ARG, "%s: temperature must be positive and finite", fn);
    if (!(top_p > 0.0f && top_p <= 1.0f))
      return fail(SPH_E_INVALID_ARG, "%s: top_p must be in (0, 1]", fn);
  }
  if (d_end > 0 && (ldh < d_end || ldw < d_end))
    return fail(SPH_E_INVALID_ARG, "%s: row strides (ldh=%lld, ldw=%lld) below d_end=%lld", fn,
                (long long)ldh, (long long)ldw, (long long)d_end);
  const int64_t k = rows_per_session - 1;
  if (!subset) return fail(SPH_E_INVALID_ARG, "%s: subset is NULL", fn);
  if (M == 0) return ok();
  if (!q || !scale) return fail(SPH_E_INVALID_ARG, "%s: q/scale is NULL", fn);
  if (d_end > 0 && !w_end) return fail(SPH_E_INVALID_ARG, "%s: w_end is NULL", fn);
  if (d_end > 0 && !codes && !h_end) return fail(SPH_E_INVALID_ARG, "%s: h_end is NULL", fn);
  if (d_end > 0 && codes && (!hq || !h_scale))
    return fail(SPH_E_INVALID_ARG, "%s: hq/h_scale is NULL", fn);
  if (k > 0 && !drafts) return fail(SPH_E_INVALID_ARG, "%s: drafts is NULL with k=%lld", fn, (long long)k);
  if (!tokens_out || !accept_len_out)
    return fail(SPH_E_INVALID_ARG, "%s: tokens_out/accept_len_out is NULL", fn);
  const int64_t n = subset->n;
  const size_t need = fuse_ws(M, n, mode) + (codes ? widen_ws(M, d_end) : 0);
  if (!workspace || ws_bytes < need)
    return fail(SPH_E_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                workspace ? ws_bytes : (size_t)0);
  if (d_end > 0 && ((reinterpret_cast<uintptr_t>(w_end) & 15) != 0 || ldw % 8 != 0 || d_end % 8 != 0))
    return fail(SPH_E_UNSUPPORTED, "%s: endpoint weight rows must be 16-byte aligned and d_end a multiple of 8",
                fn);
  if (n > (int64_t)sph::kMaxBlocks * sph::kGemvMaxIdsPerBlock)
    return fail(SPH_E_UNSUPPORTED, "%s: subset of %lld ids is too large", fn, (long long)n);
  const int64_t Kp = round_up(d_end, 8);
  const int64_t qstride = sph_payload_code_bytes(n, bits);
  const int qnb = (int)sph_payload_scale_count(n, block);

  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint64_t* best = reinterpret_cast<uint64_t*>(ws);
  // Sampling needs the whole fused row: into fused_out, else the workspace.
  float* fused = fused_out;
  if (mode == SPH_SAMPLE && !fused)
    fused = reinterpret_cast<float*>(ws + align256((size_t)M * sph::kMaxBlocks * 8));
  // int8 codes take part only where there is an endpoint partial
  const bool hcodes = codes && d_end > 0;
  const bool h_vec = d_end == 0 || hcodes ||
                     ((reinterpret_cast<uintptr_t>(h_end) & 15) == 0 && ldh % 8 == 0);
  int nblk;
  if (M > sph::kGemvMaxRows && h_vec && sph::mfma_n_tiles((int)n) <= sph::kMaxBlocks) {
    sph::MfmaArgs a{};
    a.h = static_cast<const uint16_t*>(h_end);
    a.ldh = ldh;
    if (hcodes) {
      // codes -> bf16 operands in the workspace, row scales in the epilogue
      uint16_t* wide = reinterpret_cast<uint16_t*>(ws + fuse_ws(M, n, mode));
      hipError_t e = traced("fuse_widen_codes", s, [&] {
        return sph::launch_widen_codes(hq, ldh, (int)M, (int)d_end, (int)Kp, wide, s);
      });
      if (e != hipSuccess) return hip_fail(e, "hidden-code widening launch");
      a.h = wide;
      a.ldh = Kp;
      a.hscale = h_scale;
    }
    a.M = (int)M;
    a.K = (int)d_end;
    a.w = static_cast<const uint8_t*>(w_end);
    a.ldw_bytes = ldw * 2;
    a.w_rows = subset->vocab;
    a.ids = subset->d_ids;
    a.n = (int)n;
    a.q = static_cast<const uint8_t*>(q);
    a.qstride = qstride;
    a.qscale = scale;
    a.qbits = bits;
    a.qshift = qshift;
    a.qnb = qnb;
    a.f = fused;
    a.best_part = best;
    hipError_t e = traced("fuse_mfma", s, [&] { return sph::launch_mfma(sph::kEpiFuse, 0, a, s); });
    if (e != hipSuccess) return hip_fail(e, "endpoint projection launch");
    nblk = sph::mfma_n_tiles((int)n);
  } else {
    int mr = sph::kGemvMaxRows;
    if (Kp > 0) mr = (int)std::min<int64_t>(mr, sph::kGemvLdsBytes / (Kp * 2));
    if (mr < 1) return fail(SPH_E_UNSUPPORTED, "%s: d_end=%lld too large", fn, (long long)d_end);
    const int lpr = sph::gemv_lpr((int)d_end, 0);
    const int rpi = sph::gemv_rows_per_iter(lpr);
    nblk = (int)std::min<int64_t>((n + rpi - 1) / rpi, sph::kMaxBlocks);
    for (int64_t m0 = 0; m0 < M; m0 += mr) {
      const int rows = (int)std::min<int64_t>(mr, M - m0);
      sph::GemvArgs a{};
      a.h = hcodes ? nullptr : static_cast<const uint16_t*>(h_end) + (d_end > 0 ? m0 * ldh : 0);
      a.ldh = ldh;
      if (hcodes) {
        a.hq = hq + m0 * ldh;
        a.ldhq = ldh;
        a.hscale = h_scale + m0;
      }
      a.K = (int)d_end;
      a.Kp = (int)Kp;
      a.w = static_cast<const uint8_t*>(w_end);
      a.ldw_bytes = ldw * 2;
      a.ids = subset->d_ids;
      a.n = (int)n;
      a.nblk = nblk;
      a.q = static_cast<const uint8_t*>(q) + m0 * qstride;
      a.qstride = qstride;
      a.qscale = scale + m0 * qnb;
      a.qbits = bits;
      a.qshift = qshift;
      a.qnb = qnb;
      a.f = fused ? fused + m0 * n : nullptr;
      a.best_part = best + m0 * sph::kMaxBlocks;
      hipError_t e = traced("fuse_gemv", s, [&] { return sph::launch_gemv(sph::kEpiFuse, 0, rows, a, s); });
      if (e != hipSuccess) return hip_fail(e, "endpoint projection launch");
    }
  }
  if (mode == SPH_SAMPLE) {
    hipError_t e = traced("fuse_sample", s, [&] {
      return sph::launch_sample(fused, (int)M, (int)n,
                                reinterpret_cast<const unsigned long long*>(best), nblk,
                                subset->d_ids, (int)rows_per_session, temperature, top_p, seed,
                                tokens_out, s);
    });
    if (e != hipSuccess) return hip_fail(e, "sampling launch");
    e = traced("fuse_accept", s, [&] {
      return sph::launch_accept(tokens_out, drafts, (int)n_sessions, (int)rows_per_session,
                                accept_len_out, s);
    });
    if (e != hipSuccess) return hip_fail(e, "verification launch");
    return ok();
  }
  hipError_t e = traced("fuse_final_greedy", s, [&] {
    return sph::launch_final_greedy(best, nblk, subset->d_ids, (int)n, (int)n_sessions,
                                    (int)rows_per_session, drafts, tokens_out, accept_len_out, s);
  });
  if (e != hipSuccess) return hip_fail(e, "greedy finaliser launch");
  return ok();
}

}  // namespace

int sph_fuse_verify_fmt(const void* q, const float* scale, int bits, int64_t block,
                        const void* h_end, int64_t ldh, int64_t d_end, const void* w_end,
                        int64_t ldw, sph_subset subset, int64_t n_sessions,
                        int64_t rows_per_session, const int32_t* drafts, int mode,
                        float temperature, float top_p, uint64_t seed, int32_t* tokens_out,
                        int32_t* accept_len_out, float* fused_out, void* workspace,
                        size_t ws_bytes, void* stream) {
  return fuse_verify_impl("sph_fuse_verify", false, q, scale, bits, block, h_end, nullptr, nullptr,
                          ldh, d_end, w_end, ldw, subset, n_sessions, rows_per_session, drafts,
                          mode, temperature, top_p, seed, tokens_out, accept_len_out, fused_out,
                          workspace, ws_bytes, stream);
}

int sph_fuse_verify_hq(const void* q, const float* scale, int bits, int64_t block,
                       const int8_t* hq, int64_t ldhq, const float* h_scale, int64_t d_end,
                       const void* w_end, int64_t ldw, sph_subset subset, int64_t n_sessions,
                       int64_t rows_per_session, const int32_t* drafts, int mode,
                       float temperature, float top_p, uint64_t seed, int32_t* tokens_out,
                       int32_t* accept_len_out, float* fused_out, void* workspace,
                       size_t ws_bytes, void* stream) {
  return fuse_verify_impl("sph_fuse_verify_hq", true, q, scale, bits, block, nullptr, hq, h_scale,
                          ldhq, d_end, w_end, ldw, subset, n_sessions, rows_per_session, drafts,
                          mode, temperature, top_p, seed, tokens_out, accept_len_out, fused_out,
                          workspace, ws_bytes, stream);
}

int sph_gcm_key_create(const uint8_t* key, int key_bytes, void* stream, sph_gcm_key* out) {
  if (!out) return fail(SPH_E_INVALID_ARG, "sph_gcm_key_create: out is NULL");
  *out = nullptr;
  if (!key) return fail(SPH_E_INVALID_ARG, "sph_gcm_key_create: key is NULL");
  if (key_bytes != 16 && key_bytes != 32)
    return fail(SPH_E_INVALID_ARG, "sph_gcm_key_create: key_bytes=%d not 16 or 32", key_bytes);
  std::vector<uint8_t> image;
  int nr = 0;
  if (!sph::gcm_key_setup(key, key_bytes, image, nr))
    return fail(SPH_E_INVALID_ARG, "sph_gcm_key_create: key set-up failed");
  uint8_t* d = nullptr;
  hipError_t e = hipMalloc(&d, image.size());
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(gcm key)");
  hipStream_t st = (hipStream_t)stream;
  e = hipMemcpyAsync(d, image.data(), image.size(), hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);  // the host image is freed on return
  // the image holds key material: clear the host copy
  std::fill(image.begin(), image.end(), (uint8_t)0);
  if (e != hipSuccess) {
    (void)hipFree(d);
    return hip_fail(e, "sph_gcm_key_create: upload");
  }
  *out = new sph_gcm_key_s{d, nr};
  return ok();
}

void sph_gcm_key_destroy(sph_gcm_key key) {
  if (!key) return;
  (void)hipFree(key->d_image);
  delete key;
}

size_t sph_gcm_workspace(int64_t rows, int64_t row_bytes) {
  if (rows <= 0 || row_bytes < 0) return 0;
  const int64_t n = (row_bytes + 15) / 16;
  // sized for the largest AAD, so that one workspace serves every call
  return align256((size_t)rows * (size_t)sph::gcm_parts(n, sph::kGcmMaxAad / 16, sph::gcm_chain(rows, n)) *
                  16);
}

namespace {

int gcm_call(const char* fn, bool open, sph_gcm_key key, const sph_gcm_segment* segs, int nseg,
             int64_t rows, const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes,
             uint8_t* tag, int32_t* okf, void* workspace, size_t ws_bytes, void* stream) {
  if (!key) return fail(SPH_E_INVALID_ARG, "%s: key is NULL", fn);
  if (!segs || nseg < 1 || nseg > SPH_GCM_MAX_SEGMENTS)
    return fail(SPH_E_INVALID_ARG, "%s: nseg=%d not in [1, %d] (or segments NULL)", fn, nseg,
                SPH_GCM_MAX_SEGMENTS);
  if (rows < 0 || rows > 65535) return fail(SPH_E_INVALID_ARG, "%s: rows=%lld out of range", fn, (long long)rows);
  sph::GcmSegs g{};
  g.nseg = nseg;
  int64_t row_bytes = 0;
  for (int k = 0; k < nseg; ++k) {
    const sph_gcm_segment& sg = segs[k];
    if (sg.bytes < 0 || sg.bytes > (int64_t)sph::kGcmMaxPow * 16)
      return fail(SPH_E_INVALID_ARG, "%s: segment %d has %lld bytes", fn, k, (long long)sg.bytes);
    if (sg.ld_in < sg.bytes || sg.ld_out < sg.bytes)
      return fail(SPH_E_INVALID_ARG, "%s: segment %d: row strides below the row length", fn, k);
    if (rows > 0 && sg.bytes > 0 && (!sg.in || !sg.out))
      return fail(SPH_E_INVALID_ARG, "%s: segment %d: input/output is NULL", fn, k);
    row_bytes += sg.bytes;
    g.in[k] = static_cast<const uint8_t*>(sg.in);
    g.out[k] = static_cast<uint8_t*>(sg.out);
    g.ld_in[k] = sg.ld_in;
    g.ld_out[k] = sg.ld_out;
    g.end[k] = row_bytes;
  }
  if (aad_bytes < 0 || aad_bytes > sph::kGcmMaxAad)
    return fail(SPH_E_INVALID_ARG, "%s: aad_bytes=%lld not in [0, %d]", fn, (long long)aad_bytes,
                sph::kGcmMaxAad);
  const int64_t m = (aad_bytes + 15) / 16 + (row_bytes + 15) / 16 + 1;
  if (m > sph::kGcmMaxPow)
    return fail(SPH_E_UNSUPPORTED, "%s: message of %lld bytes (+%lld AAD) exceeds %d blocks", fn,
                (long long)row_bytes, (long long)aad_bytes, sph::kGcmMaxPow);
  if (aad_bytes > 0 && ld_aad < aad_bytes)
    return fail(SPH_E_INVALID_ARG, "%s: AAD row stride below the AAD length", fn);
  if (rows == 0) return ok();
  if (!iv || !tag || (open && !okf)) return fail(SPH_E_INVALID_ARG, "%s: iv/tag/ok is NULL", fn);
  if (aad_bytes > 0 && !aad) return fail(SPH_E_INVALID_ARG, "%s: aad is NULL", fn);
  const size_t need = sph_gcm_workspace(rows, row_bytes);
  if (need > 0 && (!workspace || ws_bytes < need))
    return fail(SPH_E_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                workspace ? ws_bytes : (size_t)0);
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = traced(open ? "gcm_open" : "gcm_seal", s, [&] {
    return sph::launch_gcm(open, key->d_image, key->nr, g, (int)rows, iv,
                           static_cast<const uint8_t*>(aad), ld_aad, (int)aad_bytes, tag, okf,
                           static_cast<uint32_t*>(workspace), s);
  });
  if (e != hipSuccess) return hip_fail(e, open ? "AES-GCM open launch" : "AES-GCM seal launch");
  return ok();
}

}  // namespace

int sph_gcm_seal(sph_gcm_key key, const void* pt, int64_t ld_pt, int64_t rows, int64_t row_bytes,
                 const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes, void* ct,
                 int64_t ld_ct, uint8_t* tag, void* workspace, size_t ws_bytes, void* stream) {
  const sph_gcm_segment sg{pt, ld_pt, ct, ld_ct, row_bytes};
  return gcm_call("sph_gcm_seal", false, key, &sg, 1, rows, iv, aad, ld_aad, aad_bytes, tag, nullptr,
                  workspace, ws_bytes, stream);
}

int sph_gcm_open(sph_gcm_key key, const void* ct, int64_t ld_ct, int64_t rows, int64_t row_bytes,
                 const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes,
                 const uint8_t* tag, void* pt, int64_t ld_pt, int32_t* ok_out, void* workspace,
                 size_t ws_bytes, void* stream) {
  const sph_gcm_segment sg{ct, ld_ct, pt, ld_pt, row_bytes};
  return gcm_call("sph_gcm_open", true, key, &sg, 1, rows, iv, aad, ld_aad, aad_bytes,
                  const_cast<uint8_t*>(tag), ok_out, workspace, ws_bytes, stream);
}

int sph_gcm_seal_segments(sph_gcm_key key, const sph_gcm_segment* segments, int nseg, int64_t rows,
                          const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes,
                          uint8_t* tag, void* workspace, size_t ws_bytes, void* stream) {
  return gcm_call("sph_gcm_seal_segments", false, key, segments, nseg, rows, iv, aad, ld_aad, aad_bytes,
                  tag, nullptr, workspace, ws_bytes, stream);
}

int sph_gcm_open_segments(sph_gcm_key key, const sph_gcm_segment* segments, int nseg, int64_t rows,
                          const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes,
                          const uint8_t* tag, int32_t* ok_out, void* workspace, size_t ws_bytes,
                          void* stream) {
  return gcm_call("sph_gcm_open_segments", true, key, segments, nseg, rows, iv, aad, ld_aad, aad_bytes,
                  const_cast<uint8_t*>(tag), ok_out, workspace, ws_bytes, stream);
}

int sph_trace_start(int capacity) {
  if (capacity < 1 || capacity > (1 << 22))
    return fail(SPH_E_INVALID_ARG, "sph_trace_start: capacity %d out of range", capacity);
  std::lock_guard<std::mutex> lk(g_trace_mu);
  trace_free_locked();
  g_trace.reserve((size_t)capacity);
  for (int i = 0; i < capacity; ++i) {
    TraceSlot t{nullptr, nullptr, nullptr, false};
    hipError_t e = hipEventCreate(&t.start);
    if (e == hipSuccess) {
      e = hipEventCreate(&t.stop);
      if (e != hipSuccess) (void)hipEventDestroy(t.start);
    }
    if (e != hipSuccess) {
      trace_free_locked();
      return hip_fail(e, "sph_trace_start: hipEventCreate");
    }
    g_trace.push_back(t);
  }
  g_tracing.store(true, std::memory_order_release);
  return ok();
}

int sph_trace_stop(sph_trace_record* out, int max_records, int* n_out) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  g_tracing.store(false, std::memory_order_release);
  const size_t used = g_trace_used;
  int rc = SPH_OK;
  int k = 0;  // regions that launched a kernel
  for (size_t i = 0; i < used; ++i) {
    if (!g_trace[i].used) continue;
    hipError_t e = hipEventSynchronize(g_trace[i].stop);
    float ms = 0.0f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, g_trace[i].start, g_trace[i].stop);
    if (e != hipSuccess) {
      rc = hip_fail(e, "sph_trace_stop: reading events");
      break;
    }
    if (out && k < max_records) {
      std::memset(out[k].kernel, 0, SPH_TRACE_NAME_LEN);
      std::strncpy(out[k].kernel, g_trace[i].name, SPH_TRACE_NAME_LEN - 1);
      out[k].ms = ms;
    }
    ++k;
  }
  if (n_out) *n_out = k;
  trace_free_locked();
  return rc == SPH_OK ? ok() : rc;
}


int sph_probe_read(const void* buf, int64_t bytes, float* sink, void* stream) {
  if (!buf || !sink) return fail(SPH_E_INVALID_ARG, "sph_probe_read: buf or sink is NULL");
  if ((reinterpret_cast<uintptr_t>(buf) & 15) != 0 || bytes <= 0 || bytes % 16 != 0)
    return fail(SPH_E_INVALID_ARG, "sph_probe_read: buf must be 16-byte aligned and bytes a positive "
                                   "multiple of 16 (got %lld)", (long long)bytes);
  const hipError_t e = sph::launch_probe_read(buf, bytes, sink, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "read probe launch");
  return ok();
}

int sph_probe_mfma(int64_t iters, float* sink, void* stream, double* flops_out) {
  if (!sink || !flops_out) return fail(SPH_E_INVALID_ARG, "sph_probe_mfma: sink or flops_out is NULL");
  if (iters < 1 || iters > (int64_t(1) << 30))
    return fail(SPH_E_INVALID_ARG, "sph_probe_mfma: iters %lld not in [1, 2^30]", (long long)iters);
  const hipError_t e = sph::launch_probe_mfma((int)iters, sink, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "MFMA probe launch");
  *flops_out = sph::probe_mfma_flops(iters);
  return ok();
}

}  // extern "C"
