/*
 * speechkv.h - C ABI of the SpeechKV hot path on AMD Instinct MI355X (gfx950).
 *
 * SpeechKV (arXiv 2607.06827, "Compress the Cache, Not the Speech Embedding")
 * shortens the speech part of a speech LLM's KV cache inside the LLM.  From
 * layer l0 onward a learned linear gate scores every speech key, a softmax over
 * each non-overlapping window of w consecutive speech positions turns the
 * scores into weights, and the window's keys and values are replaced by their
 * weighted sums (Sec. III-B, Eq. 4).  Text positions are left as they are.
 * Full-resolution queries then attend over the shorter cache (Sec. III-B,
 * Eq. 5) under a mask that keeps attention causal.  At inference the pooling
 * runs once, at prefill, and decoding attends over the stored compressed cache
 * (Sec. III-C).
 *
 * Three calls carry the method:
 *   speechkv_pool_kv       prefill-time pooling into the paged cache (Eq. 4)
 *   speechkv_decode_attn   one-query-per-sequence attention over the cache (Eq. 5)
 *   speechkv_prefill_attn  full-resolution queries over the cache (Eq. 5 + mask)
 *   speechkv_pool_hidden   the same pooling applied to whole hidden states
 *                          (HS Compression, Sec. IV-A method (4))
 *   speechkv_pool_prefill_attn  pooling and prefill attention in one launch,
 *                          the pooling done on the fly (Sec. III-C)
 * and two more carry its training (Sec. III-C: the pooling runs inside the
 * forward pass and is optimised jointly with the model):
 *   speechkv_prefill_attn_bwd  gradients of speechkv_prefill_attn: dQ, dK^, dV^
 *   speechkv_pool_kv_bwd       gradients of the pooling: raw dK, dV and the
 *                              gate's du
 * Sequences with several speech runs (multi-turn inputs) take a segment table
 * instead of the one-run spans: speechkv_pool_kv_segments,
 * speechkv_prefill_attn_segments and their backward
 * speechkv_prefill_attn_bwd_segments and speechkv_pool_kv_bwd_segments.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers documented as "device" point into GPU memory of the current HIP
 *   device; pointers documented as "host" point into CPU memory.  The caller
 *   owns every buffer.  The library allocates nothing, frees nothing and
 *   never synchronises; it is safe to call from several host threads.  Its
 *   only global state is the per-device address of the static scratch of
 *   speechkv_decode_attn_noalloc, looked up once per device.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Work is enqueued asynchronously on it.
 * - Every argument is validated on the host before anything is enqueued.  A
 *   call that returns an error has enqueued nothing.  Values that live in
 *   device memory (span lengths, cache lengths, block-table entries) cannot be
 *   checked on the host: they are caller obligations listed per call.  The
 *   kernels clamp every index they derive from them, so a violation gives
 *   wrong results but no out-of-bounds access.
 * - Layers are numbered from 0.  Layer `layer` is compressed iff layer >= l0;
 *   otherwise the effective window is 1 and pooling is the identity.  (The
 *   paper numbers layers from 1: its l0 = 5, which leaves the first 4 layers
 *   at full resolution, is l0 = 4 here.)
 * - Element types: SPEECHKV_DTYPE_F32 (fp32) or SPEECHKV_DTYPE_BF16 (bf16).
 *   Arithmetic is fp32 in every kernel; results are rounded to nearest-even
 *   into the element type when stored.
 * - Supported shapes: head_dim in {64, 128}; num_q_heads = G * num_kv_heads
 *   with G in {1, 2, 4, 8}; page_size a power of two in [8, 256].
 */
#ifndef SPEECHKV_H
#define SPEECHKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes.  Every call returns SPEECHKV_OK or one negative code. */
#define SPEECHKV_OK 0
#define SPEECHKV_ERR_INVALID_ARG (-1) /* null pointer, bad size or count      */
#define SPEECHKV_ERR_UNSUPPORTED (-2) /* dtype, head_dim, G or page_size      */
#define SPEECHKV_ERR_WORKSPACE (-3)   /* workspace missing or too small       */
#define SPEECHKV_ERR_ALIAS (-4)       /* a buffer written overlaps one read or another written */
#define SPEECHKV_ERR_HIP (-5)         /* the HIP runtime refused a launch     */
#define SPEECHKV_ERR_SCRATCH (-6)     /* needs more than the static scratch   */

/* Element types. */
#define SPEECHKV_DTYPE_F32 0
#define SPEECHKV_DTYPE_BF16 1

/* Largest window size w the pooling and attention calls take, and so the
 * largest number of rows (raw_len, q_len) is INT32_MAX - SPEECHKV_MAX_WINDOW:
 * with these bounds no window count ceil(T / w) overflows 32-bit arithmetic. */
#define SPEECHKV_MAX_WINDOW 65536

/* Bytes of the static device scratch of speechkv_decode_attn_noalloc (one
 * copy per GPU, held until the process ends): 16 MiB. */
#define SPEECHKV_NOALLOC_SCRATCH_BYTES 16777216

/* Largest number of segments one sequence may have (speechkv_segments):
 * every kernel that reads a segment table scans a sequence's segments. */
#define SPEECHKV_MAX_SEGMENTS 1024

/* Mask modes for speech queries against pooled windows (Sec. III-B: each
 * query attends only to positions that precede it; the figure that draws the
 * mask is not part of the text, so two readings are offered).
 *   WINDOW_END   pooled window i becomes visible at its last frame
 *                (default: no query ever sees a frame later than itself).
 *   WINDOW_START pooled window i becomes visible at its first frame. */
#define SPEECHKV_MASK_WINDOW_END 0
#define SPEECHKV_MASK_WINDOW_START 1

/*
 * Paged KV cache of one layer (the per-layer cache of Sec. III-C).
 *
 * k_pages, v_pages  device, element type `dtype`, each laid out
 *                   [num_pages][num_kv_heads][page_size][head_dim]: one
 *                   (page, kv head) is a contiguous run of page_size rows.
 * block_table       device int32 [batch][max_pages_per_seq]; entry
 *                   (b, j) is the page that holds cache slots
 *                   [j*page_size, (j+1)*page_size) of sequence b.
 *                   Caller obligation: entries are in [0, num_pages), and no
 *                   page is shared by two sequences that one call writes.
 *                   (Entries outside that range are skipped by the kernels.)
 */
typedef struct speechkv_paged_kv {
  void* k_pages;
  void* v_pages;
  const int32_t* block_table;
  int32_t num_pages;
  int32_t page_size;
  int32_t max_pages_per_seq;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t dtype;
} speechkv_paged_kv;

/*
 * Where the speech sits inside each sequence (Sec. III-A: the LLM input is the
 * concatenation of speech and text; Sec. III-B: pooling acts on the T speech
 * positions only).  Sequence b at full resolution is
 *     [ prefix_len[b] text | speech_len[b] speech frames | suffix_len[b] text ].
 *
 * prefix_len, speech_len, suffix_len  device int32 [batch], each >= 0.
 * max_speech_len  host: an upper bound on every speech_len[b].
 * max_total_len   host: an upper bound on every prefix+speech+suffix length.
 * The two host bounds size the launch grids without a device round trip.
 * Caller obligation: the bounds hold.  (Work beyond them is not done.)
 */
typedef struct speechkv_spans {
  const int32_t* prefix_len;
  const int32_t* speech_len;
  const int32_t* suffix_len;
  int32_t max_speech_len;
  int32_t max_total_len;
} speechkv_spans;

/*
 * Sequences with several speech runs (a multi-turn input: the LLM input
 * interleaves speech and text, Sec. III-A).  Sequence b is the concatenation
 * of its segments i in [seg_start[b], seg_start[b+1]), segment i being
 *     [ text_len[i] text rows | speech_len[i] speech frames ].
 * Each speech run is pooled on its own (Eq. 4): windows of w frames start at
 * the run's first frame, and the run's last window keeps the frames it has.
 * One run [P | T | N] is the table {(P, T), (N, 0)}.
 *
 * seg_start      device int32 [batch + 1], non-decreasing, seg_start[0] >= 0,
 *                seg_start[batch] <= num_segments.
 * text_len, speech_len  device int32 [num_segments], each >= 0.
 * num_segments   host: entries in text_len and speech_len (>= 0).
 * max_segments   host: an upper bound on seg_start[b+1] - seg_start[b],
 *                0 .. SPEECHKV_MAX_SEGMENTS.
 * max_total_len  host: an upper bound on every sequence's row count.
 * Caller obligation: the bounds hold.  The kernels read at most
 * max_segments segments per sequence and at most max_total_len rows, clamp
 * every table value into range, and never read past num_segments.
 */
typedef struct speechkv_segments {
  const int32_t* seg_start;
  const int32_t* text_len;
  const int32_t* speech_len;
  int32_t num_segments;
  int32_t max_segments;
  int32_t max_total_len;
} speechkv_segments;

/*
 * speechkv_pool_kv - learned window pooling of the speech keys and values,
 * written straight into the paged cache (Sec. III-B, Eq. 4; Sec. III-C).
 *
 * For every sequence b and KV head g, with P, T, N its span lengths and
 * w_eff = (layer >= l0) ? w : 1, nW = ceil(T / w_eff):
 *   cache slot c in [0, P)          <- raw row c                (bitwise copy)
 *   cache slot P + i, i in [0, nW)  <- sum_j alpha_j * raw row j over the
 *       window j in [P + i*w_eff, min(P + (i+1)*w_eff, P + T)), where
 *       alpha = softmax_j(gate_u[g] . K[b, j, g]) over that window.  The same
 *       alpha weights the keys and the values.  A last window shorter than
 *       w_eff (T % w_eff != 0) is pooled over the frames it has.
 *   cache slot P + nW + m, m in [0, N) <- raw row P + T + m      (bitwise copy)
 * The gate of the paper is affine, g(k) = u . k + bias; the bias adds the same
 * constant to every logit of a window and cancels in the softmax, so only u
 * is taken.  With w_eff = 1 every weight is exactly 1 and the cache receives
 * the raw rows bitwise.
 *
 * k_raw, v_raw   device, element type cache->dtype.  Element (b, s, g, e) is
 *                at index b*stride_b + s*stride_s + g*stride_h + e; e (the
 *                head_dim axis) is contiguous.  Strides are in elements and
 *                must keep each row 16-byte aligned.
 * batch          number of sequences (>= 1).
 * raw_len        rows per sequence in k_raw/v_raw (>= 1).  Caller
 *                obligation: prefix+speech+suffix <= raw_len.
 * spans          host pointer to the span description.
 * w              window size R of the paper, 1 .. SPEECHKV_MAX_WINDOW.
 * gate_u         device fp32 [num_kv_heads][head_dim], the gate vector of
 *                this layer per KV head, or NULL for the zero gate (uniform
 *                averaging, the paper's initialisation).
 * layer, l0      layer index and first compressed layer (both >= 0).
 * cache          host pointer to the destination cache description.  Caller
 *                obligation: each sequence has pages for P + nW + N slots.
 * cache_len_out  device int32 [batch] receiving P + nW + N, or NULL.
 * Errors: INVALID_ARG, UNSUPPORTED, HIP; ALIAS when a page pool or
 *         cache_len_out overlaps the raw K/V byte range, the gate, the block
 *         table, the span lengths or another of the three.  UNSUPPORTED also
 *         when max_total_len * num_kv_heads * head_dim / 512 exceeds
 *         2^31 - 1 (the blocks one sequence's launch would need).
 */
int speechkv_pool_kv(const void* k_raw, const void* v_raw, int64_t stride_b,
                     int64_t stride_s, int64_t stride_h, int32_t batch,
                     int32_t raw_len, const speechkv_spans* spans, int32_t w,
                     const float* gate_u, int32_t layer, int32_t l0,
                     const speechkv_paged_kv* cache, int32_t* cache_len_out,
                     void* stream);

/*
 * speechkv_pool_kv_segments - speechkv_pool_kv for sequences with several
 * speech runs: compressed slots follow the segments in order, each text row
 * copied bitwise and each window of each run pooled with Eq. 4 as above.
 * cache_len_out receives the compressed length, the sum over the sequence's
 * segments of text_len + ceil(speech_len / w_eff).
 * Arguments as for speechkv_pool_kv, with segs (host pointer) in place of
 * spans; segs->max_total_len must not exceed raw_len.
 * Errors: INVALID_ARG, UNSUPPORTED, ALIAS, HIP.
 */
int speechkv_pool_kv_segments(const void* k_raw, const void* v_raw, int64_t stride_b,
                              int64_t stride_s, int64_t stride_h, int32_t batch,
                              int32_t raw_len, const speechkv_segments* segs, int32_t w,
                              const float* gate_u, int32_t layer, int32_t l0,
                              const speechkv_paged_kv* cache, int32_t* cache_len_out,
                              void* stream);

/*
 * speechkv_pool_hidden - learned window pooling of whole hidden states: the HS
 * Compression variant (Sec. IV-A, method (4)), which applies the pooling of
 * Eq. 4 to the entire hidden state at layer l0, so that all later layers,
 * queries included, run on the shortened sequence.  (Attention over that
 * sequence is plain causal attention: speechkv_prefill_attn and
 * speechkv_decode_attn with w = 1 over a cache built from it.)
 *
 * For every sequence b, with P, T, N its span lengths and nW = ceil(T / w):
 *   out row c in [0, P)          <- h row c                    (bitwise copy)
 *   out row P + i, i in [0, nW)  <- sum_j alpha_j * h row j over the window
 *       j in [P + i*w, min(P + (i+1)*w, P + T)), alpha = softmax_j(gate_u .
 *       h row j) over that window (a one-frame window is copied bitwise)
 *   out row P + nW + m, m in [0, N) <- h row P + T + m         (bitwise copy)
 * As in speechkv_pool_kv the gate bias cancels and only u is taken.
 *
 * h              device, element type dtype.  Element (b, s, e) is at index
 *                b*stride_b + s*stride_s + e; e (the hidden axis) is
 *                contiguous.  Strides in elements, keeping rows 16-byte aligned.
 * batch, raw_len sequences (>= 1) and rows per sequence in h (>= 1).  Caller
 *                obligation: prefix+speech+suffix <= raw_len.
 * hidden         hidden size, one of 512, 1024, 2048, 4096.
 * dtype          SPEECHKV_DTYPE_F32 or SPEECHKV_DTYPE_BF16 (h and out alike).
 * spans          host pointer to the span description.
 * w              window size, 1 .. SPEECHKV_MAX_WINDOW.
 * gate_u         device fp32 [hidden], or NULL for the zero gate.
 * out            device, [batch] sequences of out_capacity rows: element
 *                (b, c, e) at b*out_stride_b + c*out_stride_s + e.  Must not
 *                overlap h.  Rows past P + nW + N are not written.
 * out_capacity   rows per sequence in out (>= 1).  Caller obligation:
 *                out_capacity >= P + nW + N of every sequence (the compressed
 *                length, not the raw one).  Rows at or past out_capacity are
 *                never written; out_len still receives the full length, so a
 *                short buffer shows there.
 * out_len        device int32 [batch] receiving P + nW + N, or NULL.
 * Errors: INVALID_ARG, UNSUPPORTED (dtype or hidden), ALIAS (out overlaps h),
 *         HIP.
 */
int speechkv_pool_hidden(const void* h, int64_t stride_b, int64_t stride_s,
                         int32_t batch, int32_t raw_len, int32_t hidden,
                         int32_t dtype, const speechkv_spans* spans, int32_t w,
                         const float* gate_u, void* out, int64_t out_stride_b,
                         int64_t out_stride_s, int32_t out_capacity,
                         int32_t* out_len, void* stream);

/*
 * speechkv_decode_attn - one decoding step of attention over the compressed
 * cache (Sec. III-B, Eq. 5; Sec. III-C: the cache holds the pooled speech, so
 * every step reads R times fewer speech entries).
 *
 * For every sequence b and query head h (KV head g = h / G, G = num_q_heads /
 * num_kv_heads), with L = cache_len[b]:
 *   out[b, h] = sum_{c < L} softmax_c(scale * q[b, h] . K[b, c, g]) V[b, c, g]
 * Every cached slot is visible to the newest token.  If k_new and v_new are
 * given, the newest token's key and value are first stored in slot L - 1 and
 * take part in the step.  L = 0 gives out = 0.
 *
 * q, out         device, element type cache->dtype, [batch][num_q_heads][head_dim].
 * cache_len      device int32 [batch].  Caller obligations: 0 <= cache_len[b]
 *                <= max_cache_len and the sequence has pages for them.
 *                Block-table entries past a sequence's last page do not
 *                affect the result (they may hold any value).
 * max_cache_len  host bound on cache_len (sizes the split-K grid).
 * k_new, v_new   device [batch][num_kv_heads][head_dim] of cache->dtype, or
 *                both NULL.
 * scale          logit scale, finite and > 0; 1/sqrt(head_dim) in the paper.
 * num_splits     number of key ranges each (sequence, KV head) is split into
 *                (split-K); 0 selects speechkv_decode_num_splits().  With more
 *                than one split the partial results are merged by a
 *                log-sum-exp reduction in a fixed order, so results are
 *                deterministic for a given num_splits.
 * workspace      device scratch of at least
 *                speechkv_decode_workspace_bytes(...) bytes (16-byte
 *                aligned); may be NULL when that size is 0.  Its contents on
 *                entry do not matter.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, HIP; ALIAS when out or the
 * workspace overlaps q, k_new, v_new, cache_len, the block table, a page
 * pool or each other, or (with k_new given, so the pools are written) when a
 * page pool overlaps q, k_new, v_new, cache_len, the block table or the
 * other pool.
 */
int speechkv_decode_attn(const void* q, int32_t batch, int32_t num_q_heads,
                         const speechkv_paged_kv* cache,
                         const int32_t* cache_len, int32_t max_cache_len,
                         const void* k_new, const void* v_new, float scale,
                         int32_t num_splits, void* out, void* workspace,
                         size_t workspace_bytes, void* stream);

/*
 * speechkv_decode_attn_noalloc - speechkv_decode_attn for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops and
 * harnesses that forbid hipMalloc).  Same arguments, results and errors as
 * speechkv_decode_attn, bit for bit, except that there is no workspace: the
 * split partials go to a static device array of
 * SPEECHKV_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs
 * on, until the process ends.
 *
 * - The call allocates and frees nothing.  The first call on a device looks
 *   up that device's copy of the array (with the device current) and keeps
 *   its address; later calls reuse it.
 * - Every call on one GPU shares that GPU's array, and the array keeps the
 *   last call's contents.  Nothing in it has to start at zero: every split
 *   writes its whole partial before the merge reads it.  Calls that overlap
 *   in time on one GPU (different streams, or host threads without ordering)
 *   race on the array and give wrong results; order them on one stream.
 * - SPEECHKV_ERR_SCRATCH: the step needs more than
 *   SPEECHKV_NOALLOC_SCRATCH_BYTES of split partials
 *   (speechkv_decode_workspace_bytes(...) above it).  The automatic split
 *   count (num_splits = 0) never does: it keeps the split grid at about 1024
 *   blocks, whose partials take at most 8.5 MiB.  Nothing is enqueued.
 * - SPEECHKV_ERR_HIP: the device's array could not be looked up.
 */
int speechkv_decode_attn_noalloc(const void* q, int32_t batch, int32_t num_q_heads,
                                 const speechkv_paged_kv* cache,
                                 const int32_t* cache_len, int32_t max_cache_len,
                                 const void* k_new, const void* v_new, float scale,
                                 int32_t num_splits, void* out, void* stream);

/*
 * speechkv_prefill_attn - full-resolution queries over the compressed cache,
 * causal over the compressed sequence (Sec. III-B, Eq. 5 and the mask that
 * follows it; Sec. III-C: the same computation is applied on the fly during
 * training).
 *
 * Query row p of sequence b is full-resolution position p, p in [0, P+T+N).
 * Key c of the compressed sequence (length P + nW + N, as written by
 * speechkv_pool_kv) becomes visible at position tau(c):
 *   prefix key c < P             tau = c
 *   pooled key P + i             tau = last frame of window i  (WINDOW_END)
 *                                tau = first frame of window i (WINDOW_START)
 *   suffix key P + nW + m        tau = P + T + m
 * and row p attends to the keys with tau(c) <= p.  tau is increasing in c, so
 * each row sees a prefix of the cache.  A row that sees no key (for example a
 * speech row before the first window closes when P = 0) gets out = 0 and
 * lse = -inf.  With w_eff = 1 this is ordinary causal attention.
 *
 * q, out         device, element type cache->dtype,
 *                [batch][q_len][num_q_heads][head_dim], dense.  Rows
 *                p >= P+T+N of a sequence are neither read nor written.
 * q_len          rows allocated per sequence (>= max_total_len).
 * spans, w, layer, l0  as for speechkv_pool_kv (they define nW and tau).
 * mask_mode      SPEECHKV_MASK_WINDOW_END or SPEECHKV_MASK_WINDOW_START.
 * scale          logit scale, finite and > 0; 1/sqrt(head_dim) in the paper.
 * lse            device fp32 [batch][num_q_heads][q_len] receiving the
 *                natural-log log-sum-exp of each row's scaled logits, or NULL.
 * Errors: INVALID_ARG, UNSUPPORTED, HIP; ALIAS when out or lse overlaps q, a
 *         page pool, the block table, the span lengths or each other.
 */
int speechkv_prefill_attn(const void* q, int32_t batch, int32_t num_q_heads,
                          int32_t q_len, const speechkv_paged_kv* cache,
                          const speechkv_spans* spans, int32_t w, int32_t layer,
                          int32_t l0, int32_t mask_mode, float scale, void* out,
                          float* lse, void* stream);

/*
 * speechkv_prefill_attn_segments - speechkv_prefill_attn for sequences with
 * several speech runs (the cache written by speechkv_pool_kv_segments).  A
 * text key is visible from its own row, a pooled window of any run from its
 * last frame (WINDOW_END) or its first frame (WINDOW_START); the position a
 * key becomes visible at still grows with the key, so each row sees a prefix
 * of the cache.
 * Arguments as for speechkv_prefill_attn, with segs (host pointer) in place
 * of spans; segs->max_total_len must not exceed q_len.
 * Errors: INVALID_ARG, UNSUPPORTED, ALIAS, HIP.
 */
int speechkv_prefill_attn_segments(const void* q, int32_t batch, int32_t num_q_heads,
                                   int32_t q_len, const speechkv_paged_kv* cache,
                                   const speechkv_segments* segs, int32_t w, int32_t layer,
                                   int32_t l0, int32_t mask_mode, float scale, void* out,
                                   float* lse, void* stream);

/*
 * speechkv_pool_prefill_attn - speechkv_pool_kv followed by
 * speechkv_prefill_attn in one launch: the attention reads the raw keys and
 * values and pools each key tile on the fly (Sec. III-C: in training the
 * pooling of Eq. 4 runs inside the forward pass), and the pooled rows are
 * stored into the paged cache as well, so that decoding (or the backward)
 * can follow.
 *
 * The cache, cache_len_out, out and lse receive exactly what the two calls
 * would write, bit for bit: the pooled rows come from the same arithmetic,
 * and the attention over them is the same.  Every pooled row is stored once,
 * also rows that no query sees.
 *
 * q, out, q_len, num_q_heads, mask_mode, scale, lse  as for
 *                speechkv_prefill_attn.
 * k_raw, v_raw, stride_b, stride_s, stride_h, raw_len, w, gate_u, layer, l0,
 * cache_len_out  as for speechkv_pool_kv; max_total_len must not exceed
 *                raw_len or q_len.
 * cache          host pointer to the cache description; written as by
 *                speechkv_pool_kv.  dtype must be SPEECHKV_DTYPE_BF16.
 * Nothing written (the pages, out, lse) may overlap anything read (q, the raw
 * K/V, the gate) or another written buffer (ALIAS).
 * Errors: INVALID_ARG, UNSUPPORTED (also for fp32), ALIAS, HIP.
 */
int speechkv_pool_prefill_attn(const void* q, int32_t batch, int32_t num_q_heads,
                               int32_t q_len, const void* k_raw, const void* v_raw,
                               int64_t stride_b, int64_t stride_s, int64_t stride_h,
                               int32_t raw_len, const speechkv_spans* spans, int32_t w,
                               const float* gate_u, int32_t layer, int32_t l0,
                               const speechkv_paged_kv* cache, int32_t* cache_len_out,
                               int32_t mask_mode, float scale, void* out, float* lse,
                               void* stream);

/*
 * speechkv_prefill_attn_bwd - gradients of speechkv_prefill_attn with respect
 * to the queries and the compressed keys and values (training, Sec. III-C;
 * the chain rule of Eq. 5 under the same mask).
 *
 * Given the forward's inputs, its output `out` and log-sum-exp `lse`, and the
 * gradient `dout` of the output, with P = softmax(scale q k^T) over the keys
 * each row sees:
 *   Delta_p = dout_p . out_p,  dZ = P o (dout v^T - Delta)
 *   dq = scale dZ k^,  dk^ = scale dZ^T q,  dv^ = P^T dout
 * (key gradients summed over the query heads of each KV head).  P is
 * recomputed from lse; nothing of size rows x keys is stored.
 *
 * q, out, dout   device, element type cache->dtype,
 *                [batch][q_len][num_q_heads][head_dim], dense.
 * lse            device fp32 [batch][num_q_heads][q_len], as the forward wrote it.
 * cache, spans, w, layer, l0, mask_mode, scale  as for the forward call.
 * dq             device, element type cache->dtype, layout of q.  Rows
 *                p >= P+T+N are not written; a row that sees no key gets 0.
 * dk_hat, dv_hat device fp32 [batch][hat_capacity][num_kv_heads][head_dim]:
 *                row c of sequence b is the gradient of cache slot c.  Rows
 *                c >= min(P+nW+N, hat_capacity) are not written.  Caller
 *                obligation: hat_capacity >= P+nW+N for the full gradient.
 * workspace      device, >= speechkv_prefill_attn_bwd_workspace_bytes bytes,
 *                16-byte aligned; receives Delta.
 * Nothing written may overlap an input or another output (ALIAS).
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, ALIAS, HIP.
 */
int speechkv_prefill_attn_bwd(const void* q, int32_t batch, int32_t num_q_heads,
                              int32_t q_len, const speechkv_paged_kv* cache,
                              const speechkv_spans* spans, int32_t w,
                              int32_t layer, int32_t l0, int32_t mask_mode,
                              float scale, const void* out, const float* lse,
                              const void* dout, void* dq, float* dk_hat,
                              float* dv_hat, int32_t hat_capacity,
                              void* workspace, size_t workspace_bytes,
                              void* stream);

/*
 * speechkv_prefill_attn_bwd_segments - speechkv_prefill_attn_bwd for
 * sequences with several speech runs (the forward's
 * speechkv_prefill_attn_segments); segs (host pointer) replaces spans and
 * segs->max_total_len must not exceed q_len.  Everything else as above.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, ALIAS, HIP.
 */
int speechkv_prefill_attn_bwd_segments(const void* q, int32_t batch, int32_t num_q_heads,
                                       int32_t q_len, const speechkv_paged_kv* cache,
                                       const speechkv_segments* segs, int32_t w,
                                       int32_t layer, int32_t l0, int32_t mask_mode,
                                       float scale, const void* out, const float* lse,
                                       const void* dout, void* dq, float* dk_hat,
                                       float* dv_hat, int32_t hat_capacity, void* workspace,
                                       size_t workspace_bytes, void* stream);

/* Workspace bytes of speechkv_prefill_attn_bwd (one fp32 per query row and
 * head), or 0 for invalid arguments.  Host only. */
size_t speechkv_prefill_attn_bwd_workspace_bytes(int32_t batch,
                                                 int32_t num_q_heads,
                                                 int32_t q_len);

/*
 * speechkv_pool_kv_bwd - gradients of speechkv_pool_kv with respect to the
 * raw keys, the raw values and the gate vectors (training, Sec. III-C; the
 * chain rule of Eq. 4).
 *
 * For window i of sequence b, KV head g, with frames j, logits s_j = u_g . k_j
 * and alpha = softmax_j(s):
 *   dalpha_j = dk^_i . k_j + dv^_i . v_j
 *   ds_j = alpha_j (dalpha_j - sum_j' alpha_j' dalpha_j')
 *   dk_j = alpha_j dk^_i + ds_j u_g,   dv_j = alpha_j dv^_i
 *   du_g = sum over sequences, windows and frames of ds_j k_j
 * A text row (and a one-frame window) was copied: its gradient is that of the
 * slot it became.  With w_eff = 1 every raw row gets its slot's gradient and
 * du = 0.
 *
 * k_raw, v_raw   device, element type dtype, strides as for speechkv_pool_kv.
 * num_kv_heads, head_dim  the raw tensors' heads (at most 65535) and head
 *                size (64 or 128); otherwise UNSUPPORTED.
 * spans, w, gate_u, layer, l0  as for the forward call (gate_u NULL: zero gate).
 * dk_hat, dv_hat device fp32 [batch][hat_capacity][num_kv_heads][head_dim],
 *                e.g. from speechkv_prefill_attn_bwd.  Caller obligation:
 *                hat_capacity >= P+nW+N (slots at or past it count as 0).
 * dk_raw, dv_raw device, element type dtype, the strides of k_raw: receive
 *                the gradients of rows [0, P+T+N); other rows are not written.
 * du             device fp32 [num_kv_heads][head_dim] receiving the gate
 *                gradient, or NULL to skip it.
 * workspace      device, >= speechkv_pool_kv_bwd_workspace_bytes bytes,
 *                16-byte aligned, when du is not NULL (per-block partial sums,
 *                added in a fixed order: the result is deterministic).
 * Nothing written may overlap an input or another output (ALIAS).
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, ALIAS, HIP.
 */
int speechkv_pool_kv_bwd(const void* k_raw, const void* v_raw,
                         int64_t stride_b, int64_t stride_s, int64_t stride_h,
                         int32_t batch, int32_t raw_len, int32_t num_kv_heads,
                         int32_t head_dim, int32_t dtype,
                         const speechkv_spans* spans, int32_t w,
                         const float* gate_u, int32_t layer, int32_t l0,
                         const float* dk_hat, const float* dv_hat,
                         int32_t hat_capacity, void* dk_raw, void* dv_raw,
                         float* du, void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * speechkv_pool_kv_bwd_segments - speechkv_pool_kv_bwd for sequences with
 * several speech runs (the forward's speechkv_pool_kv_segments); segs (host
 * pointer) replaces spans and segs->max_total_len must not exceed raw_len.
 * The workspace size is speechkv_pool_kv_bwd_workspace_bytes with
 * max_total_len = segs->max_total_len.  Everything else as above.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, ALIAS, HIP.
 */
int speechkv_pool_kv_bwd_segments(const void* k_raw, const void* v_raw,
                                  int64_t stride_b, int64_t stride_s, int64_t stride_h,
                                  int32_t batch, int32_t raw_len, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t dtype,
                                  const speechkv_segments* segs, int32_t w,
                                  const float* gate_u, int32_t layer, int32_t l0,
                                  const float* dk_hat, const float* dv_hat,
                                  int32_t hat_capacity, void* dk_raw, void* dv_raw,
                                  float* du, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* Workspace bytes of speechkv_pool_kv_bwd with a gate gradient, for
 * max_total_len = spans->max_total_len, or 0 for invalid or unsupported
 * arguments.  Host only. */
size_t speechkv_pool_kv_bwd_workspace_bytes(int32_t batch, int32_t max_total_len,
                                            int32_t num_kv_heads,
                                            int32_t head_dim);

/* Length of the compressed sequence, P + ceil(T / w_eff) + N (Sec. III-B,
 * Sec. III-C), or -1 for a negative length, w < 1 or negative layer/l0.
 * Host only. */
int64_t speechkv_compressed_len(int32_t prefix_len, int32_t speech_len,
                                int32_t suffix_len, int32_t w, int32_t layer,
                                int32_t l0);

/* Compressed length of one sequence given as segments (host arrays of
 * num_segments entries), or -1 for a negative length or count, w < 1, a
 * negative layer or l0. */
int64_t speechkv_compressed_len_segments(const int32_t* text_len, const int32_t* speech_len,
                                         int32_t num_segments, int32_t w, int32_t layer,
                                         int32_t l0);

/* Split count chosen by speechkv_decode_attn when num_splits = 0: the power
 * of two, at most 32, that minimises an estimate of the launch time from the
 * number of (sequence, KV head) pairs and the longest cache (a split costs a
 * merge launch, so short caches and large batches stay whole, long caches of
 * few sequences are split; every split keeps at least 64 keys).  Host only;
 * returns -1 on a non-positive batch/num_kv_heads or a negative length. */
int32_t speechkv_decode_num_splits(int32_t batch, int32_t num_kv_heads,
                                   int32_t max_cache_len);

/* Bytes of workspace speechkv_decode_attn needs for num_splits splits
 * (0 = the automatic choice), or 0 when no workspace is needed.  Host only;
 * returns 0 for invalid arguments (the decode call reports those). */
size_t speechkv_decode_workspace_bytes(int32_t batch, int32_t num_q_heads,
                                       int32_t num_kv_heads, int32_t head_dim,
                                       int32_t max_cache_len,
                                       int32_t num_splits);

/* Static text for a status code.  Host only; never NULL. */
const char* speechkv_status_string(int status);

/* Library version string, e.g. "0.1.0".  Host only. */
const char* speechkv_version(void);

#ifdef __cplusplus
} /* extern "C" */
#endif

#endif /* SPEECHKV_H */
