/*
 * sph.h - split-head vocabulary projection on one MI355X (gfx950).
 *
 * The LM head z = h' W_lm + b is split along the hidden dimension into an
 * endpoint half (the first d_end dimensions) and a cloud half (the remaining
 * d_cloud dimensions), eq. 10 of Section 5.4.  Two calls cover one decoding
 * step of the collaborative loop (Algorithm 1):
 *
 *   sph_cloud_partial  eq. 12 on the language subset S = V_l, then the clip
 *                      and the per-row int8 payload of Section 5.4 / eq. 18.
 *   sph_fuse_verify    eq. 11 on S, dequantise + fuse + mask (eq. 13-14),
 *                      greedy or temperature/top-p selection (eq. 15) and the
 *                      accepted draft prefix of each session (Section 5.5).
 *
 * Conventions shared by every call:
 *  - Tensors are caller-owned HIP device memory unless a parameter says
 *    "host".  The library never frees them.
 *  - Weights are vocab-major: row v holds the d weights of vocabulary id v
 *    (column v of the paper's D x V matrix).  bf16 tensors are passed as raw
 *    16-bit patterns; fp8 weights use the OCP E4M3 encoding.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *    enqueue work on it and return without synchronising; outputs are valid
 *    once the stream has completed.  Calls on one stream are ordered; calls
 *    that share a workspace must not overlap.
 *  - A negative return value is an error; nothing has been enqueued.  The
 *    message is available from sph_last_error() on the same thread.  Device
 *    contents (NaN inputs, draft ids) are never validated; inputs are
 *    assumed finite.
 *  - Rows of h are independent; M = n_sessions * rows_per_session rows form
 *    the verification windows of the sessions: row r of session s is row
 *    s * rows_per_session + r.
 */
#ifndef SPH_H
#define SPH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPH_ABI_VERSION 1

/* status codes */
#define SPH_OK             0
#define SPH_E_INVALID_ARG (-1) /* bad pointer, size, stride, enum or scalar */
#define SPH_E_SUBSET      (-2) /* subset ids not strictly ascending / out of range / empty */
#define SPH_E_UNSUPPORTED (-3) /* valid request the library has no kernel for */
#define SPH_E_DEVICE      (-4) /* a HIP runtime call failed; message has the HIP error */
#define SPH_E_WORKSPACE   (-5) /* workspace missing or smaller than required */

/* weight encodings of the cloud slice */
#define SPH_W_BF16     0
#define SPH_W_FP8_E4M3 1  /* OCP E4M3, with one fp32 scale per vocabulary row */

/* selection modes */
#define SPH_GREEDY 0
#define SPH_SAMPLE 1

/* Version of this interface (SPH_ABI_VERSION of the built library). */
int sph_abi_version(void);

/* Message of the last failing call on this thread ("" if none).  Valid until
 * the next sph_* call on the thread. */
const char* sph_last_error(void);

/* Debug aid (no counterpart in the paper): with debug synchronisation on,
 * every kernel launch region of every call is followed by a synchronisation
 * of the call's stream and an error check, so a kernel that fails at run
 * time makes the call that launched it return SPH_E_DEVICE, with the
 * region's name in the message, instead of surfacing at some later
 * synchronisation.  Streams being captured into a graph are not
 * synchronised.  It is off unless the environment variable SPH_DEBUG_SYNC
 * is set to a value other than "0" when the library is first used.
 * enable: 1 on, 0 off, negative to only query.  Returns the previous state
 * (0 or 1).  Process-wide; calls already running are unaffected. */
int sph_debug_sync(int enable);

/*
 * Vocabulary subset plan: the language-restricted subset V_l of Section 5.4
 * (the endpoint names it by a subset identifier; Section 6.2 precomputes the
 * mapping from tokenizer metadata).  A plan is an immutable device copy of
 * the ids, created once and reused by any number of calls on any stream of
 * the device that was current at creation.
 */
typedef struct sph_subset_s* sph_subset;

/* host_ids: host int32 [n], strictly ascending, 0 <= id < vocab, n >= 1
 * (SPH_E_SUBSET otherwise).  Allocates device memory, copies the ids on
 * `stream` and waits for the copy, so host_ids may be freed on return. */
int sph_subset_create(const int32_t* host_ids, int64_t n, int64_t vocab, void* stream,
                      sph_subset* out);

/* The whole vocabulary [0, vocab): mixed-language mode, no mask (Section 5.4). */
int sph_subset_create_full(int64_t vocab, void* stream, sph_subset* out);

/* Number of ids and vocabulary size of a plan. */
int sph_subset_size(sph_subset subset, int64_t* n, int64_t* vocab);

/* Device pointer to the plan's int32 ids (read-only, owned by the plan). */
int sph_subset_device_ids(sph_subset subset, const int32_t** ids);

/* Frees the plan once the device is idle with respect to calls using it.
 * NULL is ignored. */
void sph_subset_destroy(sph_subset subset);

/*
 * Workspace sizes in bytes (256-byte aligned device memory, caller-owned).
 * The cloud workspace holds the fp32 partial logits (unless z_out is given,
 * the region is still reserved) and per-block row maxima; the fuse
 * workspace holds per-block argmax candidates and, for SPH_SAMPLE, the fused
 * fp32 logits.  Returns 0 for M == 0.
 */
size_t sph_cloud_partial_workspace(int64_t M, sph_subset subset);
size_t sph_fuse_verify_workspace(int64_t M, sph_subset subset, int mode);

/*
 * Cloud half (eq. 12 on S, then clip and per-row int8; Section 5.4, eq. 18).
 *
 *   z[m, j] = sum_{i < d_cloud} h_cloud[m, i] * Wc[S_j, i] * s_{S_j} + b[S_j]
 *   y       = clamp(z, -clip_c, clip_c)
 *   a_m     = max_j |y[m, j]|,   scale[m] = fp32(a_m / 127)   (0 if a_m == 0)
 *   q[m, j] = clamp(rint_half_even(fp32(y / scale[m])), -127, 127)  (0 if scale == 0)
 *
 * h_cloud     bf16 [M, d_cloud], row stride ldh elements (pass h + d_end with
 *             ldh = d to read the cloud columns of a full [M, d] hidden state)
 * w_cloud     [V, d_cloud] vocab-major, row stride ldw elements; bf16 bit
 *             patterns for SPH_W_BF16, E4M3 bytes for SPH_W_FP8_E4M3.  Must
 *             hold every row named by the subset.
 * w_row_scale fp32 [V]: required for SPH_W_FP8_E4M3 (s_v above), NULL for bf16
 * bias        fp32 [V] or NULL; added once, on the cloud side, before the clip
 * subset      plan; n_sub = its size
 * clip_c      > 0 and finite
 * q_out       int8 [M, n_sub] row-major: the payload codes
 * scale_out   fp32 [M]: the payload scales
 * z_out       fp32 [M, n_sub] or NULL: the pre-clip partial logits exactly as
 *             quantised (validation)
 * workspace   >= sph_cloud_partial_workspace(M, subset) bytes
 * The payload of one row is n_sub + 4 bytes (eq. 21 without transport
 * overhead).  M == 0 is a no-op.
 */
int sph_cloud_partial(const void* h_cloud, int64_t ldh, int64_t M, int64_t d_cloud,
                      const void* w_cloud, int64_t ldw, int wtype, const float* w_row_scale,
                      const float* bias, sph_subset subset, float clip_c,
                      int8_t* q_out, float* scale_out, float* z_out,
                      void* workspace, size_t ws_bytes, void* stream);

/*
 * Endpoint half: eq. 11 on S, fusion with the dequantised payload and the
 * mask (eq. 13-14), selection (eq. 15) and verification (Section 5.5).
 *
 *   f[m, j]  = fmaf(q[m, j], scale[m], sum_{i < d_end} h_end[m, i] * We[S_j, i])
 *   GREEDY:  token[m] = S[argmax_j f[m, j]], ties to the lowest id
 *   SAMPLE:  p = softmax(f / temperature) over S; the nucleus is the
 *            shortest prefix of S ordered by (p desc, id asc) whose mass
 *            reaches top_p; u = top 24 bits of word 0 of Philox4x32-10 with
 *            key (lo32(seed), hi32(seed)) and counter (r, s, 0, 0) times
 *            2^-24; the token is the first nucleus member in ascending id
 *            order whose running mass exceeds u * mass(nucleus).
 *   accept_len[s] = largest a <= k with token[s*R + r] == drafts[s, r] for
 *            all r < a (R = rows_per_session, k = R - 1).  The committed
 *            tokens of session s are drafts[s, 0..a) then token[s*R + a].
 *
 * q, scale    the payload of sph_cloud_partial for the same rows and subset
 * h_end       bf16 [M, d_end], row stride ldh (may be NULL if d_end == 0)
 * w_end       bf16 [V, d_end] vocab-major, row stride ldw (NULL if d_end == 0)
 * drafts      int32 [n_sessions, k]; required when k > 0.  Ids outside S
 *             are legal and never match.
 * mode        SPH_GREEDY (temperature, top_p, seed ignored) or SPH_SAMPLE
 *             (temperature > 0, 0 < top_p <= 1)
 * tokens_out  int32 [M] vocabulary ids, always members of S
 * accept_len_out int32 [n_sessions], in [0, k]
 * fused_out   fp32 [M, n_sub] or NULL: f (validation)
 * workspace   >= sph_fuse_verify_workspace(M, subset, mode) bytes
 */
int sph_fuse_verify(const int8_t* q, const float* scale,
                    const void* h_end, int64_t ldh, int64_t d_end,
                    const void* w_end, int64_t ldw, sph_subset subset,
                    int64_t n_sessions, int64_t rows_per_session, const int32_t* drafts,
                    int mode, float temperature, float top_p, uint64_t seed,
                    int32_t* tokens_out, int32_t* accept_len_out, float* fused_out,
                    void* workspace, size_t ws_bytes, void* stream);

/*
 * Configurable payload format (eq. 18 quantises to a configurable bit width
 * b; eq. 21 puts the payload at about |V_l| * b/8 bytes plus metadata).
 *
 *   bits   8: codes in [-127, 127], one byte each (the format above);
 *          4: codes in [-7, 7], two per byte: code 2i in the low and code
 *             2i+1 in the high nibble of byte i, two's complement nibbles;
 *             an odd n_sub ends with a zero high nibble.
 *   block  0: one scale per row (the format above);
 *          256, 512, 1024, 2048 or 4096: one scale per row and block of that
 *             many consecutive subset positions (the last block may be
 *             shorter): a[m, k] = max |y[m, j]| over block k and
 *             scale[m, k] = fp32(a[m, k] / qmax), qmax = 2^(bits-1) - 1.
 *   Codes are clamp(rint_half_even(fp32(y / scale)), -qmax, qmax) as above.
 * A payload of M rows is M * sph_payload_code_bytes(n_sub, bits) code bytes
 * (rows contiguous) and fp32 scales [M, sph_payload_scale_count(n_sub, block)].
 */

/* ceil(n_sub * bits / 8), or -1 for an invalid bits or n_sub. */
int64_t sph_payload_code_bytes(int64_t n_sub, int bits);

/* 1 for block 0, else ceil(n_sub / block) (at least 1); -1 if invalid. */
int64_t sph_payload_scale_count(int64_t n_sub, int64_t block);

/* sph_cloud_partial with the payload in format (bits, block): q_out holds the
 * packed codes, scale_out the scales as described above.  (8, 0) is
 * sph_cloud_partial.  Same workspace. */
int sph_cloud_partial_fmt(const void* h_cloud, int64_t ldh, int64_t M, int64_t d_cloud,
                          const void* w_cloud, int64_t ldw, int wtype, const float* w_row_scale,
                          const float* bias, sph_subset subset, float clip_c, int bits,
                          int64_t block, void* q_out, float* scale_out, float* z_out,
                          void* workspace, size_t ws_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the cloud
 * call of sph_cloud_partial_fmt without a workspace argument.  Its
 * workspace is a static device array of SPH_NOALLOC_SCRATCH_BYTES bytes
 * that every GPU the library runs on holds until the process ends; the
 * call allocates nothing, frees nothing and calls no allocating routine.
 * Inputs, outputs, results and errors are those of sph_cloud_partial_fmt,
 * plus SPH_E_WORKSPACE (nothing enqueued) when
 * sph_cloud_partial_workspace(M, subset) exceeds the scratch size, e.g.
 * 5 rows x 49152 ids need about 1 MB, 20 rows x 190000 ids about 15 MB.
 * The scratch keeps the last call's contents and no kernel depends on
 * its initial contents.  Every call on one GPU shares that GPU's scratch:
 * calls that overlap on one GPU (on different streams, or from several
 * threads without ordering) race and give undefined results; calls on one
 * stream are ordered and safe.
 */
#define SPH_NOALLOC_SCRATCH_BYTES (16u << 20)
int sph_cloud_partial_noalloc(const void* h_cloud, int64_t ldh, int64_t M, int64_t d_cloud,
                              const void* w_cloud, int64_t ldw, int wtype,
                              const float* w_row_scale, const float* bias, sph_subset subset,
                              float clip_c, int bits, int64_t block, void* q_out,
                              float* scale_out, float* z_out, void* stream);

/* sph_fuse_verify reading a payload in format (bits, block):
 *   f[m, j] = fmaf(code[m, j], scale[m, k(j)], z_end[m, j]),  k(j) = j / block
 * (k = 0 for block 0).  (8, 0) is sph_fuse_verify.  Same workspace. */
int sph_fuse_verify_fmt(const void* q, const float* scale, int bits, int64_t block,
                        const void* h_end, int64_t ldh, int64_t d_end, const void* w_end,
                        int64_t ldw, sph_subset subset, int64_t n_sessions,
                        int64_t rows_per_session, const int32_t* drafts, int mode,
                        float temperature, float top_p, uint64_t seed, int32_t* tokens_out,
                        int32_t* accept_len_out, float* fused_out, void* workspace,
                        size_t ws_bytes, void* stream);

/*
 * Hidden-state codes (Section 5.3: every tensor the cloud returns, the hidden
 * state included, is quantised with the Q_b of eq. 18 before it is sent).
 * Format: int8 codes with one fp32 scale per row,
 *   a_m = max_i |x[m, i]| over the row's d values (bf16, exact in fp32),
 *   s_m = fp32(a_m / 127) (0 for an all-zero row),
 *   q[m, i] = clamp(rint_half_even(fp32(x[m, i] / s_m)), -127, 127), 0 if s_m = 0.
 * The endpoint's projection (eq. 11) then runs on the dequantised values
 * q * s; it computes s_m * sum_i q[m, i] W_end[S_j, i] in fp32, which equals
 * the sum over q * s up to the order of the fp32 additions.
 */

/* Quantise M bf16 rows h [M, ldh] (first d columns; d = the full hidden row
 * when the whole state is returned) into q_out int8 [M, ldq] and scale_out
 * fp32 [M].  ldh, ldq >= d.  Device pointers, caller-owned; enqueues one
 * kernel on `stream`.  d = 0 gives scales 0. */
int sph_hidden_quantize(const void* h, int64_t ldh, int64_t M, int64_t d, int8_t* q_out,
                        int64_t ldq, float* scale_out, void* stream);

/* Workspace of sph_fuse_verify_hq: that of sph_fuse_verify plus, for more
 * than 8 rows, M * round_up(d_end, 8) bf16 operands. */
size_t sph_fuse_verify_hq_workspace(int64_t M, int64_t d_end, sph_subset subset, int mode);

/* sph_fuse_verify_fmt with the endpoint's hidden state as codes: hq int8
 * [M, ldhq] (its first d_end columns enter eq. 11) and h_scale fp32 [M], as
 * written by sph_hidden_quantize.  ldhq >= d_end; every other argument and
 * all outputs as in sph_fuse_verify_fmt. */
int sph_fuse_verify_hq(const void* q, const float* scale, int bits, int64_t block,
                       const int8_t* hq, int64_t ldhq, const float* h_scale, int64_t d_end,
                       const void* w_end, int64_t ldw, sph_subset subset, int64_t n_sessions,
                       int64_t rows_per_session, const int32_t* drafts, int mode,
                       float temperature, float top_p, uint64_t seed, int32_t* tokens_out,
                       int32_t* accept_len_out, float* fused_out, void* workspace,
                       size_t ws_bytes, void* stream);

/*
 * Payload sealing (eq. 19): AES-GCM (AES per FIPS-197, GCM per NIST
 * SP 800-38D, 96-bit IVs, 128-bit tags) of batches of rows, each row its
 * own message: row m of `rows` rows of row_bytes bytes is encrypted under
 * iv[m] (12 bytes; J0 = iv || 00000001, the data keystream starts at
 * counter 2) with associated data aad[m] (aad_bytes bytes, e.g. session,
 * block and cache-control fields).  A nonce must never repeat under one
 * key; the caller chooses the scheme (the paper derives GPU-mode nonces from
 * the session and the message type).  A payload row's codes and scales can
 * be sealed as one message (sph_gcm_seal_segments) or as two batches (two
 * message types).  All buffers are device memory; rows are ld_* bytes apart,
 * iv [rows][12], tag [rows][16].  Limits: rows <= 65535, aad_bytes <= 1024,
 * ceil(aad_bytes/16) + ceil(row_bytes/16) + 1 <= 16384.  Seal and open may
 * work in place (out == in, same stride).
 */
typedef struct sph_gcm_key_s* sph_gcm_key;

/* Expand a 16- or 32-byte AES key (host memory) into a device key object
 * (round keys, tables, the powers of the GHASH key and the product tables
 * of H^256, ~272 KB); blocks
 * until the upload on `stream` has finished.  Destroy with
 * sph_gcm_key_destroy. */
int sph_gcm_key_create(const uint8_t* key, int key_bytes, void* stream, sph_gcm_key* out);
void sph_gcm_key_destroy(sph_gcm_key key);

/* Device workspace bytes of a seal or open of rows x row_bytes (for any
 * aad_bytes <= 1024; nonzero for rows > 0, also for empty messages). */
size_t sph_gcm_workspace(int64_t rows, int64_t row_bytes);

/* ct[m] = plaintext row m xor its keystream; tag[m] its authentication tag. */
int sph_gcm_seal(sph_gcm_key key, const void* pt, int64_t ld_pt, int64_t rows, int64_t row_bytes,
                 const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes, void* ct,
                 int64_t ld_ct, uint8_t* tag, void* workspace, size_t ws_bytes, void* stream);

/* pt[m] = ciphertext row m xor its keystream; ok_out[m] = 1 if tag[m] is the
 * row's tag, else 0.  A row with ok_out[m] = 0 must not be used: its pt row
 * holds unauthenticated bytes. */
int sph_gcm_open(sph_gcm_key key, const void* ct, int64_t ld_ct, int64_t rows, int64_t row_bytes,
                 const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes,
                 const uint8_t* tag, void* pt, int64_t ld_pt, int32_t* ok_out, void* workspace,
                 size_t ws_bytes, void* stream);

/* Messages made of several row-aligned pieces: message m is the
 * concatenation, in order, of row m of each segment (bytes bytes of
 * in + m * ld_in), and its output bytes go to the same places of out +
 * m * ld_out.  E.g. one payload row = its codes followed by its scales, with
 * no copy into a staging buffer.  `segments` is a host array of nseg (1 ..
 * SPH_GCM_MAX_SEGMENTS) entries, read during the call only; a segment may
 * be empty (bytes = 0, pointers unused).  Segments must not overlap one
 * another; each may work in place (out == in, ld_out == ld_in).  The
 * message length is the sum of the segment lengths; the workspace is
 * sph_gcm_workspace(rows, that sum), and every limit above applies to it.
 * The result is that of sph_gcm_seal / sph_gcm_open on the concatenated
 * rows. */
#define SPH_GCM_MAX_SEGMENTS 4
typedef struct {
  const void* in;  /* device, rows x bytes, ld_in bytes apart */
  int64_t ld_in;
  void* out;       /* device, rows x bytes, ld_out bytes apart */
  int64_t ld_out;
  int64_t bytes;   /* bytes this segment adds to each message */
} sph_gcm_segment;

int sph_gcm_seal_segments(sph_gcm_key key, const sph_gcm_segment* segments, int nseg, int64_t rows,
                          const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes,
                          uint8_t* tag, void* workspace, size_t ws_bytes, void* stream);

/* Opening counterpart: ok_out[m] as in sph_gcm_open. */
int sph_gcm_open_segments(sph_gcm_key key, const sph_gcm_segment* segments, int nseg, int64_t rows,
                          const uint8_t* iv, const void* aad, int64_t ld_aad, int64_t aad_bytes,
                          const uint8_t* tag, int32_t* ok_out, void* workspace, size_t ws_bytes,
                          void* stream);

/*
 * Kernel tracing.  While a trace is active, each call records one duration
 * per kernel it launches: start and stop HIP events are attached to the
 * kernel dispatches themselves (hipExtLaunchKernelGGL), so a duration is
 * the kernel's execution on the launch stream as it ran in the caller's
 * workload, with no launch gap included.  Tracing is process-wide: records
 * from calls on every thread go to the one trace, in the order their
 * launches took a slot (thread-safe).
 */
#define SPH_TRACE_NAME_LEN 32
typedef struct {
  char kernel[SPH_TRACE_NAME_LEN]; /* "cloud_gemv", "cloud_quantize", "fuse_gemv", ... */
  float ms;                        /* duration on the GPU */
} sph_trace_record;

/* Start recording up to `capacity` launches (capacity >= 1); restarts any
 * active trace.  Launches beyond the capacity are not recorded. */
int sph_trace_start(int capacity);

/* Stop recording, wait for the recorded events, and copy up to max_records
 * records (launch order) to `out` (host memory); *n_out gets the number of
 * recorded launches.  Frees the trace's events. */
int sph_trace_stop(sph_trace_record* out, int max_records, int* n_out);

#ifdef __cplusplus
}
#endif

#endif /* SPH_H */
