/*
 * mw.h -- C ABI of the block-causal attention library for MI355X (gfx950).
 *
 * Operations (from "MiniWorld: Democratizing the Training of Video World
 * Models from Scratch"):
 *   - block-causal multi-head self-attention, forward and backward
 *     (Sec. 3.2, "Block-Causal Video DiT"): the token sequence is split into
 *     temporally ordered chunks of chunk_len tokens; a token attends to every
 *     token of its own chunk and of all earlier chunks, never to later chunks;
 *   - the rolling KV cache of committed chunks and the attention of queued
 *     in-flight chunks over it (Sec. 3.5, "Streaming Inference",
 *     "Structured Rolling KV Cache", "Pipelined Denoising").
 *
 * Conventions (every entry point):
 *   - Tensors are device pointers to contiguous row-major arrays, except in
 *     the *_strided entry points, which take [B, H, T, D] views described by
 *     mw_strides (the head dimension D contiguous).  bf16 means
 *     IEEE bfloat16 stored as 16-bit words.  Every pointer must be 16-byte
 *     aligned.  The caller allocates and owns every buffer, including the
 *     backward workspace; the library never allocates or frees device memory.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the legacy default
 *     stream) and the call returns without waiting.  Faults during kernel
 *     execution surface at the caller's next synchronisation.  Only kernel
 *     launches are enqueued (no memset, copy or allocation), so the attention
 *     calls and mw_quantize_fp8 may be recorded into a HIP graph; the
 *     mw_kvcache_* calls that change a ring's host descriptor (init, append,
 *     evict, set_sink, rope_shift) must run outside it, and a recorded
 *     attention call keeps the ring state (window, pending re-shifts) it was
 *     recorded with.
 *   - Arguments are validated before anything is enqueued; on error nothing
 *     is enqueued, no state changes, and a negative mw_status is returned.
 *     mw_last_error() then describes the problem (per-thread message).
 *   - No C++ exception crosses this boundary.  Calls are reentrant, except
 *     that one mw_kvcache must not be used by two threads at once.
 */
#ifndef MW_H
#define MW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void* mw_stream_t; /* a hipStream_t */

typedef enum {
  MW_OK = 0,
  MW_EINVAL = -1,        /* null pointer, non-positive size, inconsistent sizes */
  MW_EUNSUPPORTED = -2,  /* head dimension other than 64, 72 or 128, or a limit exceeded */
  MW_EALIGN = -3,        /* a pointer that is not 16-byte aligned */
  MW_EFULL = -4,         /* append to a ring whose slots are all live */
  MW_EEMPTY = -5,        /* evict more chunks than are live */
  MW_EHIP = -6           /* the HIP runtime reported an error at launch */
} mw_status;

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* mw_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int mw_version(void);

/* Element strides of a bf16 [B, H, T, D] tensor view whose D elements are
 * contiguous: element (b, h, t, d) is at base + b*b + h*h + t*t + d (in
 * elements).  A contiguous [B, H, T, D] tensor has {H*T*D, T*D, D}; a
 * [B, T, H, D] tensor (the layout of a QKV projection's output) seen as
 * [B, H, T, D] has {T*H*D, D, H*D}; q, k, v inside one fused [B, T, 3, H, D]
 * tensor have {3*T*H*D, D, 3*H*D}.  Requirements, checked before anything is
 * enqueued: every stride a multiple of 8 (16-byte aligned rows; MW_EALIGN),
 * b and h >= 0, t >= D (MW_EINVAL); a view that is written (an output) must
 * not overlap itself (MW_EINVAL).  Inputs may overlap one another; outputs
 * must not overlap inputs or other outputs (not checked). */
typedef struct {
  int64_t b, h, t;
} mw_strides;

/* Largest supported window (committed chunks attended to) and queued-chunk count. */
#define MW_MAX_WINDOW 64
#define MW_MAX_QUEUED 64
/* Largest ring of an e4m3 cache (its per-slot re-shift record, below). */
#define MW_MAX_SLOTS 128

/* ------------------------------------------------------------------------
 * Training: block-causal attention (Sec. 3.2).
 *
 * Query row i and key j (0-based positions in the sequence) lie in chunks
 * floor(i/chunk_len) and floor(j/chunk_len); key j is visible to row i iff
 * floor(j/chunk_len) <= floor(i/chunk_len).  T need not be a multiple of
 * chunk_len (the last chunk is then shorter).  With S = scale * Q K^T masked
 * to -inf on hidden pairs:
 *     O   = softmax(S) V                          (row-wise softmax)
 *     LSE = log(sum_j exp(S_ij)) over visible j   (natural log)
 *
 * q, k, v, o : bf16 [B, H, T, D]
 * lse        : fp32 [B, H, T]  (needed by the backward pass)
 * D          : 64, 72 or 128.  scale > 0 (the usual choice is 1/sqrt(D)).
 * Arithmetic: bf16 products, fp32 accumulation and softmax; the softmax
 * probabilities are rounded to bf16 before the product with V; O is rounded
 * to bf16 (nearest even).
 * Errors: MW_EINVAL (null pointer, B/H/T/chunk_len < 1, scale <= 0),
 * MW_EALIGN, MW_EUNSUPPORTED (D), MW_EHIP.
 * ---------------------------------------------------------------------- */
int mw_block_causal_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                             int B, int H, int T, int D, int chunk_len, float scale,
                             mw_stream_t stream);

/* The same on strided views, so that q, k, v can be read (and o written) in
 * the layout the projections use, with no transposing copy.
 * strides: 4 entries, for q, k, v, o in that order (NULL = all contiguous).
 * lse stays contiguous fp32 [B, H, T].  Errors: as above, plus the stride
 * checks of mw_strides. */
int mw_block_causal_attn_fwd_strided(const void* q, const void* k, const void* v, void* o, float* lse,
                                     const mw_strides* strides, int B, int H, int T, int D, int chunk_len,
                                     float scale, mw_stream_t stream);

/* Bytes of device workspace mw_block_causal_attn_bwd needs (fp32 row terms). */
size_t mw_block_causal_attn_bwd_workspace_size(int B, int H, int T, int D);

/* Backward of the forward above for the loss sum(dO * O): the analytic softmax
 * gradient
 *     dV = P^T dO,  dP = dO V^T,  Delta_i = sum_d dO_id O_id,
 *     dS = P * (dP - Delta),  dQ = scale dS K,  dK = scale dS^T Q,
 * with P recomputed from q, k and the forward's lse.
 *
 * q, k, v, o, d_o : bf16 [B, H, T, D] (o and lse from mw_block_causal_attn_fwd)
 * lse             : fp32 [B, H, T]
 * dq, dk, dv      : bf16 [B, H, T, D], written (not accumulated)
 * workspace       : device buffer of at least
 *                   mw_block_causal_attn_bwd_workspace_size(B, H, T, D) bytes;
 *                   its contents on entry do not matter.
 * The result is deterministic (no atomics).
 * Errors: as the forward, plus MW_EINVAL if workspace_bytes is too small.
 */
int mw_block_causal_attn_bwd(const void* q, const void* k, const void* v, const void* o,
                             const void* d_o, const float* lse, void* dq, void* dk, void* dv,
                             void* workspace, size_t workspace_bytes,
                             int B, int H, int T, int D, int chunk_len, float scale,
                             mw_stream_t stream);

/* The backward on strided views.  strides: 8 entries, for q, k, v, o, d_o, dq,
 * dk, dv in that order (NULL = all contiguous); lse and the workspace stay
 * contiguous.  Errors: as above, plus the stride checks of mw_strides. */
int mw_block_causal_attn_bwd_strided(const void* q, const void* k, const void* v, const void* o,
                                     const void* d_o, const float* lse, void* dq, void* dk, void* dv,
                                     void* workspace, size_t workspace_bytes, const mw_strides* strides,
                                     int B, int H, int T, int D, int chunk_len, float scale,
                                     mw_stream_t stream);

/* The backward above (contiguous tensors) with no workspace argument, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation.  The row terms
 * (8 bytes per row) live in a 32 MiB device array inside the library, one
 * copy per GPU, held until the process ends; so B * H * T must not exceed
 * 4,194,304 (MW_EUNSUPPORTED beyond).  The call allocates and frees nothing.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (other streams, other host threads) race, and the caller must serialise
 * them.  Nothing has to be cleared between calls: every row term is written
 * before it is read.  The calling thread's current device must be the device
 * of the stream and of the tensors.  Arguments, layout, arithmetic and result
 * as mw_block_causal_attn_bwd.
 * Errors: as mw_block_causal_attn_bwd, plus MW_EUNSUPPORTED above the row
 * limit and MW_EHIP if the array's device address cannot be obtained. */
int mw_block_causal_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o,
                                     const void* d_o, const float* lse, void* dq, void* dk, void* dv,
                                     int B, int H, int T, int D, int chunk_len, float scale,
                                     mw_stream_t stream);

/* ------------------------------------------------------------------------
 * Rolling KV cache (Sec. 3.5, "Structured Rolling KV Cache").
 *
 * Committed chunks enter a FIFO of capacity S chunks kept as a ring of S
 * slots over caller-owned device buffers k_slots and v_slots, each bf16
 * [S, B, H, L, D].  Chunks are numbered by commit order c = 0, 1, ...; head
 * counts commits and tail counts evictions, so the live chunks are
 * [tail, head) and chunk c lives in slot c mod S.  A committed chunk's keys
 * and values are never modified afterwards.  The struct is plain data: it can
 * be copied to snapshot the ring state and restored by copying it back
 * (together with the slot buffers' contents).
 * ---------------------------------------------------------------------- */
typedef struct {
  void* k_slots;
  void* v_slots;
  int S, B, H, L, D;
  int64_t head;        /* chunks committed so far */
  int64_t tail;        /* chunks evicted so far  */
  const void* k_sink;  /* sink anchor (see mw_kvcache_set_sink), or NULL */
  const void* v_sink;
  int sink_len;        /* sink tokens (0: no sink) */
  int elem_bytes;      /* 2: bf16 slots (mw_kvcache_init); 1: e4m3 slots (mw_kvcache_init_fp8) */
  float k_scale;       /* e4m3 slots: key value = code * k_scale (1 for bf16 slots) */
  float v_scale;       /* e4m3 slots: value value = code * v_scale (1 for bf16 slots) */
  /* RoPE re-shift record of e4m3 slots, whose keys are rotated when a call
   * loads them instead of in place (see mw_kvcache_rope_shift); all zero for
   * bf16 slots. */
  int64_t rope_total;  /* sum of the shifts applied so far */
  int rope_offset;     /* band of those shifts: dim_offset, dim_count and theta of the */
  int rope_count;      /* first one (later shifts must use the same band) */
  float rope_theta;
  int rope_set;        /* 1 once a band is recorded */
  int64_t rope_at_commit[MW_MAX_SLOTS]; /* rope_total when the chunk in each slot was committed */
} mw_kvcache;

/* Initialise an empty ring over k_slots/v_slots (bf16 [S,B,H,L,D]), without a
 * sink; no device work.
 * Errors: MW_EINVAL (null, sizes < 1), MW_EALIGN, MW_EUNSUPPORTED (D not 64, 72 or 128). */
int mw_kvcache_init(mw_kvcache* c, void* k_slots, void* v_slots, int S, int B, int H, int L, int D);

/* Sink anchor (Sec. 3.5): the initial clean context kept permanently, outside
 * the FIFO.  k_sink, v_sink: caller-owned bf16 [B, H, sink_len, D] (the cache
 * keeps the pointers, not a copy; the caller keeps them alive and unchanged).
 * The sink comes first in the key sequence of mw_chunk_attn_cached, is visible
 * to every queued chunk, is never evicted and is not re-shifted.  sink_len = 0
 * (pointers ignored) removes it.  Host only.
 * Errors: MW_EINVAL (null cache, sink_len < 0, null pointers with sink_len > 0),
 * MW_EALIGN, MW_EUNSUPPORTED (sink_len too large). */
int mw_kvcache_set_sink(mw_kvcache* c, const void* k_sink, const void* v_sink, int sink_len);

/* Rotary position embedding on one band of the head dimension: dimensions
 * [dim_offset, dim_offset + dim_count) form dim_count/2 interleaved pairs
 * (2i, 2i+1); pair i at position p is rotated by p * theta^(-2i/dim_count). */
typedef struct {
  int dim_offset; /* even, >= 0 */
  int dim_count;  /* even, 2..128, dim_offset + dim_count <= D */
  float theta;    /* > 0, e.g. 10000 */
} mw_rope;

/* RoPE re-shifting (Sec. 3.5): rotate the keys of every live committed chunk
 * (not the sink) by -shift positions on the rope band, so the retained window
 * is re-indexed from the start after `shift` positions of history were evicted
 * (shift = evicted chunks x positions per chunk).  Relative positions inside
 * the window are unchanged; values are untouched.
 * bf16 slots are rotated in place (the paper's first option): bf16 in, fp32
 * rotation (cos/sin computed on the host in double), bf16 out (nearest even);
 * shift = 0 or no live chunk: no device work.
 * e4m3 slots are rotated on load (the paper's second option), since rotating
 * 8-bit keys in place would re-round them at every shift: this call only adds
 * shift to c->rope_total (host only, no device work); a chunk's keys are kept
 * as committed, and mw_chunk_attn_cached_fp8 rotates each window chunk by
 * -(rope_total - its rope_at_commit) positions when it loads the window (one
 * rounding to e4m3 per call, none accumulated over shifts).  The band and
 * theta of an e4m3 cache's first shift are recorded; later shifts must use the
 * same ones.
 * Errors: MW_EINVAL (null cache or rope, invalid band, theta <= 0, a band or
 * theta other than the recorded one of an e4m3 cache), MW_EHIP. */
int mw_kvcache_rope_shift(mw_kvcache* c, int shift, const mw_rope* rope, mw_stream_t stream);

/* Commit one chunk: enqueue a copy of k_chunk and v_chunk (bf16 [B,H,L,D]) into
 * slot head mod S, then head += 1 (host state changes at call time).  An e4m3
 * cache also records rope_at_commit[slot] = rope_total.
 * Errors: MW_EINVAL, MW_EALIGN, MW_EFULL (head - tail == S), MW_EHIP. */
int mw_kvcache_append(mw_kvcache* c, const void* k_chunk, const void* v_chunk, mw_stream_t stream);

/* Commit from strided [B, H, L, D] views (e.g. K and V straight out of a
 * [B, L, H, D] projection); the slot itself is contiguous.  strides: 2
 * entries, for k_chunk and v_chunk (NULL = contiguous).  Errors: as above,
 * plus the stride checks of mw_strides. */
int mw_kvcache_append_strided(mw_kvcache* c, const void* k_chunk, const void* v_chunk,
                              const mw_strides* strides, mw_stream_t stream);

/* Discard the n_chunks oldest live chunks (tail += n_chunks).  Host only.
 * Errors: MW_EINVAL (null, n_chunks < 0), MW_EEMPTY (n_chunks > head - tail). */
int mw_kvcache_evict(mw_kvcache* c, int n_chunks);

/* Number of live chunks (head - tail), or a negative mw_status for a null cache. */
int mw_kvcache_live(const mw_kvcache* c);

/* Slot holding logical chunk `chunk` if it is live, else -1 (also for a null cache). */
int mw_kvcache_slot_of(const mw_kvcache* c, int64_t chunk);

/* ------------------------------------------------------------------------
 * Cached chunk attention for the pipelined denoiser (Sec. 3.5).
 *
 * n_queued in-flight chunks of q_len tokens each attend to the sink anchor
 * (if set), the `window` newest live committed chunks (window = -1: all live
 * chunks) and the in-flight chunks' own keys.  The keys form the virtual sequence
 *   [sink (sink_len tokens)] ++ [window chunks, oldest first (window * L tokens)]
 *   ++ [queued chunks 0..n_queued-1]
 * and queued chunk j sees
 *   MW_QUEUED_CAUSAL  : the sink, the window and queued chunks 0..j (the
 *                       committed history plus the preceding chunks of the
 *                       active window; the chunk-wise causal rule of Sec. 3.5);
 *   MW_QUEUED_ISOLATED: the sink, the window and itself only.
 *
 * q, k_new, v_new, o : bf16 [B, H, n_queued*q_len, D] with B, H, D those of the cache
 * lse                : fp32 [B, H, n_queued*q_len] or NULL
 * workspace          : optional device buffer.  With at least
 *                      mw_chunk_attn_cached_workspace_size(...) bytes the key
 *                      range of each query tile is split over several
 *                      workgroups (fp32 partial results in the workspace, then a
 *                      merge), which keeps the GPU busy when there are few query
 *                      tiles (few or short queued chunks); the heaviest query
 *                      tiles may run unsplit while the lighter ones, which run
 *                      last, are split (mw_chunk_attn_cached_plan).  NULL or a
 *                      smaller buffer: a plan that fits (possibly no split).
 *                      The result does not depend on the plan beyond fp32
 *                      rounding.
 * Keys are visited in logical order whatever the ring offset, so the result
 * for a given window content does not depend on where the ring wrapped.
 * Errors: MW_EINVAL (null pointers, n_queued/q_len < 1, window > live,
 * window < -1, unknown flags, scale <= 0), MW_EALIGN,
 * MW_EUNSUPPORTED (window > MW_MAX_WINDOW or n_queued > MW_MAX_QUEUED), MW_EHIP.
 * ---------------------------------------------------------------------- */
enum { MW_QUEUED_CAUSAL = 0, MW_QUEUED_ISOLATED = 1 };

/* Workspace bytes that let mw_chunk_attn_cached use its preferred split plan
 * for this shape under either visibility rule (0 when neither would split).
 * For an e4m3 cache, also the rotated window keys of mw_chunk_attn_cached_fp8's
 * rotation on load (window * B * H * L * 128 bytes, rounded up to 256), needed
 * only while shifts are pending but always included.  Negative window: all
 * live. */
size_t mw_chunk_attn_cached_workspace_size(const mw_kvcache* c, int n_queued, int q_len, int window);

/* The key-range split plan that mw_chunk_attn_cached (mw_chunk_attn_cached_fp8
 * for an e4m3 cache) uses for this shape, visibility rule (flags) and
 * workspace size (0: no workspace): *n_splits key ranges for the lighter
 * query tiles of each head, of which the *n_whole heaviest (the last) run
 * unsplit; *n_splits = 1 means no split and then *n_whole = 0.  The plan comes
 * from a cost model of the kernel's dispatch and does not change the result
 * beyond fp32 rounding.  Host-only: no device work.
 * Errors: MW_EINVAL (null pointers, n_queued/q_len < 1, window < -1 or above
 * the live chunks, unknown flags), MW_EUNSUPPORTED (as mw_chunk_attn_cached). */
int mw_chunk_attn_cached_plan(const mw_kvcache* c, int n_queued, int q_len, int window, int flags,
                              size_t workspace_bytes, int* n_splits, int* n_whole);

int mw_chunk_attn_cached(const void* q, const void* k_new, const void* v_new,
                         int n_queued, int q_len, const mw_kvcache* c, int window, int flags,
                         void* o, float* lse, float scale, void* workspace, size_t workspace_bytes,
                         mw_stream_t stream);

/* Cached chunk attention on strided [B, H, n_queued*q_len, D] views of q,
 * k_new, v_new and o.  strides: 4 entries in that order (NULL = contiguous);
 * lse, the ring and the sink keep their layouts.  Errors: as above, plus the
 * stride checks of mw_strides. */
int mw_chunk_attn_cached_strided(const void* q, const void* k_new, const void* v_new,
                                 int n_queued, int q_len, const mw_kvcache* c, int window, int flags,
                                 void* o, float* lse, float scale, void* workspace, size_t workspace_bytes,
                                 const mw_strides* strides, mw_stream_t stream);

/* ------------------------------------------------------------------------
 * fp8 inference variant: quantized cached chunk attention.
 *
 * The paper names quantization as a way to cut the cost of streaming
 * inference (Sec. 6, "Efficient deployment").  This variant stores the
 * committed window, the sink and the queued chunks' Q, K, V as OCP e4m3
 * (1 sign, 4 exponent bits with bias 7, 3 mantissa bits; finite range
 * +-448; no infinities) with per-tensor scales, value = code * scale, and
 * computes the cached chunk attention of Sec. 3.5 (same key sequence and
 * visibility rules as mw_chunk_attn_cached) with both products in e4m3 on the
 * matrix cores: scores and softmax statistics in fp32, the probabilities
 * (at most 2^8 by construction) rounded to e4m3 (nearest even) before the PV
 * product, O normalised in fp32 and stored as bf16.  Head dimension 128 only.
 * ---------------------------------------------------------------------- */

/* Quantize a bf16 [B, H, T, D] view (strides as in mw_strides; NULL =
 * contiguous) into a contiguous e4m3 [B, H, T, D] tensor y (1 byte per
 * element): code = RNE_e4m3(clamp(fl32(x * fl32(1 / scale)), -448, 448)),
 * where fl32 is fp32 rounding (nearest even) and 1/scale is computed on the
 * host in fp32.  x must be finite (non-finite values saturate).  D: a multiple
 * of 8 (64, 72 or 128).  y must be 16-byte aligned and must not overlap x.
 * Errors: MW_EINVAL (null, sizes < 1, scale not finite and > 0), MW_EALIGN,
 * MW_EUNSUPPORTED (D), MW_EHIP. */
int mw_quantize_fp8(const void* x, const mw_strides* x_strides, void* y, int B, int H, int T, int D,
                    float scale, mw_stream_t stream);

/* Initialise an empty ring whose slots hold e4m3 K and V: k_slots, v_slots are
 * e4m3 [S, B, H, L, D] (1 byte per element), with per-tensor scales k_scale,
 * v_scale (> 0, finite) fixed for the cache's lifetime.  mw_kvcache_append and
 * mw_kvcache_append_strided take bf16 chunks and quantize them into the slot
 * with these scales (mw_quantize_fp8's rounding).  The sink
 * (mw_kvcache_set_sink) must be e4m3 [B, H, sink_len, D] quantized with the
 * same scales.  mw_kvcache_rope_shift records shifts for rotation on load
 * (see there).  mw_chunk_attn_cached rejects an e4m3 cache (MW_EINVAL); use
 * mw_chunk_attn_cached_fp8.  Eviction, live counts and slot numbering are
 * those of the bf16 ring.  No device work.
 * Errors: MW_EINVAL (null, sizes < 1, bad scales), MW_EALIGN,
 * MW_EUNSUPPORTED (D other than 128, S > MW_MAX_SLOTS). */
int mw_kvcache_init_fp8(mw_kvcache* c, void* k_slots, void* v_slots, int S, int B, int H, int L, int D,
                        float k_scale, float v_scale);

/* Cached chunk attention over an e4m3 cache (mw_kvcache_init_fp8).
 * q8, k8_new, v8_new : e4m3 [B, H, n_queued*q_len, 128], contiguous; q8
 *                      quantized with q_scale, k8_new and v8_new with the
 *                      cache's k_scale and v_scale (mw_quantize_fp8)
 * o                  : bf16 [B, H, n_queued*q_len, 128] view (o_strides, NULL =
 *                      contiguous); lse: fp32 [B, H, n_queued*q_len] or NULL
 * scale              : softmax scale applied to the dequantized scores
 * The scores are (q8 . k8) * q_scale * k_scale * scale, the output
 * sum_j p_j v8_j * v_scale / sum_j p_j.  window, flags, workspace (size from
 * mw_chunk_attn_cached_workspace_size on the e4m3 cache) as in
 * mw_chunk_attn_cached.
 * Rotation on load: when a window chunk has shifts pending (rope_total !=
 * its rope_at_commit), every window chunk's keys are used rotated by
 * -(rope_total - rope_at_commit[slot]) positions on the recorded band: each
 * pair is decoded, rotated in fp32 (cos/sin of the angle computed in double),
 * clamped to +-448 and rounded to e4m3 (nearest even); the slots are not
 * modified.  Calls with one query tile per head (at most 256 queued rows)
 * whose key ranges span few window chunks (chunks of at least 64 keys)
 * rotate each K tile as the attention kernel stages it; the others first
 * write the rotated window keys to the start of the workspace and the
 * attention reads them from there.
 * Both routes give the same bytes.  Either way the call reserves
 * window * B * H * L * 128 bytes of workspace (rounded up to 256) before the
 * key-range partials; mw_chunk_attn_cached_workspace_size of an e4m3 cache
 * always includes them.
 * Errors: as mw_chunk_attn_cached, plus MW_EINVAL for a bf16 cache, q_scale
 * not finite and > 0, or shifts pending with a workspace too small for the
 * rotated window keys. */
int mw_chunk_attn_cached_fp8(const void* q8, const void* k8_new, const void* v8_new, int n_queued, int q_len,
                             const mw_kvcache* c, int window, int flags, void* o, float* lse, float scale,
                             float q_scale, void* workspace, size_t workspace_bytes, const mw_strides* o_strides,
                             mw_stream_t stream);

/* ------------------------------------------------------------------------
 * Pipelined denoising schedule (Sec. 3.5, "Pipelined Denoising" and the
 * latent update of Eq. 7; non-decreasing chunk timesteps, Eq. 4; timestep
 * shift, Eq. 6).  Host-only planning of the streaming loop: which chunks are
 * in flight at each tick (one DiT pass over the active window), their noise
 * levels and updates, and which chunks are committed, evicted and re-shifted
 * afterwards.  No device work and no state: a tick's plan is a function of the
 * configuration and the tick number.
 *
 * Chunks are numbered 0 .. n_chunks-1 in generation order.  `stride` new
 * chunks enter per tick at tau = 1 (fewer at the end of the stream); each
 * stays U = floor(window / stride) ticks and gets one update per tick, so the
 * window never holds more than U * stride <= window chunks.  Before its k-th
 * update a chunk is at tau = g(k/U), g(x) = shift(1 - x),
 * shift(t) = s t / (1 + (s - 1) t); its update is g((k+1)/U) - g(k/U) <= 0
 * and its last update lands on tau = 0 exactly, after which it is committed
 * (Delta-tau allocated from the stride and the window so that every chunk
 * reaches the data endpoint before commit).  With n_bins > 0 each level is
 * rounded to the nearest multiple of 1/n_bins.  Older chunks are never noisier
 * than newer ones (Eq. 4).  After the tick's commits the FIFO keeps the newest
 * cache_chunks committed chunks; the evicted chunks' frames are the RoPE
 * re-shift of the retained keys.  Positions are frames of the re-indexed
 * sequence [sink (sink_frames) | cached chunks | in-flight chunks].
 * ---------------------------------------------------------------------- */
typedef struct {
  int window;           /* in-flight chunk capacity, 1 .. MW_MAX_QUEUED */
  int stride;           /* chunks entering per tick, 1 .. window */
  int n_chunks;         /* chunks to generate, >= 1 */
  int cache_chunks;     /* capacity of the committed FIFO, >= 0 */
  int frames_per_chunk; /* latent frames (RoPE positions) per chunk, >= 1 */
  int sink_frames;      /* frames of the sink anchor, >= 0 */
  double shift;         /* timestep shift s > 0 (1: none) */
  int n_bins;           /* 0, or the number of discrete timestep bins */
} mw_sched_config;

typedef struct {
  int64_t tick;
  int first;             /* oldest in-flight chunk; in flight: first .. first+n_active-1 */
  int n_active;          /* in-flight chunks this tick (n_queued of mw_chunk_attn_cached) */
  int updates_per_chunk; /* U */
  double tau[MW_MAX_QUEUED];  /* noise level of each in-flight chunk before this tick's update */
  double dtau[MW_MAX_QUEUED]; /* its update (<= 0); unused entries are 0 */
  int n_commit;          /* chunks first .. first+n_commit-1 reach tau = 0 and are committed, in order */
  int n_evict;           /* oldest cached chunks evicted after the commits */
  int rope_shift;        /* frames the retained keys move back: n_evict * frames_per_chunk */
  int cache_live;        /* cached chunks after this tick */
  int pos_first;         /* frame of the oldest in-flight chunk during this tick */
} mw_sched_tick;

/* Ticks until every chunk is committed (floor((n_chunks-1)/stride) + U), or a
 * negative mw_status for an invalid configuration (MW_EINVAL, MW_EUNSUPPORTED). */
int64_t mw_sched_num_ticks(const mw_sched_config* cfg);

/* Plan of tick `tick` (0-based) into *out.  Errors: MW_EINVAL (invalid
 * configuration, NULL out), MW_EUNSUPPORTED, MW_EEMPTY (tick out of range). */
int mw_sched_plan(const mw_sched_config* cfg, int64_t tick, mw_sched_tick* out);

#ifdef __cplusplus
}
#endif
#endif /* MW_H */
