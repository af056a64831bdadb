/*
 * voxzip.h -- C ABI of libvoxzip.so, the MI355X (gfx950) hot path of VoxZip
 * ("Semantic-Anchored Temporal KV Cache Compression for Long-Context Audio
 * Inference", arXiv 2608.08569).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers are DEVICE pointers unless marked [host].  The caller owns all
 *    memory; the library allocates nothing and keeps no state between calls
 *    (thread-safe as long as concurrent calls do not share buffers).
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL
 *    is the default stream).  Errors found on the host are returned before any
 *    work is queued; a failed launch returns VZ_ERR_HIP.
 *  - KV caches are [n_layers][kv_heads][cap][d], contiguous in d.  The element
 *    type of q, k, v, caches and outputs is `dtype` (VZ_F32 or VZ_BF16);
 *    scores are float32 [n_layers][cap]; positions are int32 [n_layers][cap].
 *    All layers hold the same number of resident tokens `len`.
 *  - Supported shapes: d in {64, 128}; n_q_heads a multiple of kv_heads with
 *    n_q_heads / kv_heads <= 16; every size positive and every index below 2^31.
 *  - Slots are not kept in position order: each slot carries its logical
 *    position in `pos`, and the sink and recent windows are defined on
 *    positions.  Positions inside one layer must be distinct.
 */
#ifndef VOXZIP_H
#define VOXZIP_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define VZ_API __attribute__((visibility("default")))
#else
#define VZ_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define VZ_OK 0
#define VZ_ERR_INVALID -1     /* a null pointer, a bad scalar (gamma, budget, windows) */
#define VZ_ERR_SHAPE -2       /* inconsistent sizes (n_q_heads % kv_heads, d, counts) */
#define VZ_ERR_CAPACITY -3    /* the cache or an output has no room */
#define VZ_ERR_UNSUPPORTED -4 /* dtype / head size / group size the library does not serve */
#define VZ_ERR_HIP -5         /* a HIP call failed; voxzip_last_error() has its text */
#define VZ_ERR_WORKSPACE -6   /* workspace missing, not 16-byte aligned, or smaller than voxzip_workspace_bytes() */
#define VZ_IDLE 1             /* per-sequence status of a ragged call: an idle batch slot (cap[s] == 0), skipped */

/* Element types. */
#define VZ_F32 0
#define VZ_BF16 1

/* Operations whose workspace can be queried. */
#define VZ_OP_DECODE 1
#define VZ_OP_EVICT 2
#define VZ_OP_DECODE_EVICT 3   /* voxzip_decode_evict */

/*
 * Stage-1 span offsets (Sec. 3.2.1: confidence filter, Eq. 3 time-to-token
 * map, uniform partition of each semantic interval into groups, background
 * tokens kept one per span).  Host function: every pointer is a host pointer.
 *
 *  t_start_ms, t_end_ms  int64 [n_seg] segment times in ms (clipped to
 *               [0, t_total_ms]); conf float32 [n_seg]; text_len int32 [n_seg]
 *               (text tokens of each segment).
 *  t_total_ms   duration of the audio, > 0; L_a audio tokens, >= 0.
 *  conf_threshold  a segment is used when conf > conf_threshold (0.3 in the paper).
 *  off_out      int32 [L_a + 1] (room for the worst case): receives span_off
 *               for voxzip_fuse_spans, off_out[0] = 0, strictly increasing,
 *               off_out[*n_spans_out] = L_a.
 *  n_spans_out  receives the number of spans.
 * A segment covers tokens [floor(L_a t_start / t_total), floor(L_a t_end /
 * t_total)) (exact integer arithmetic).  Segments are taken in the order
 * (first token, last token, input order); a segment starting inside tokens
 * already covered starts where they end; an empty interval, or a segment
 * with text_len < 1, is skipped.  An interval of n tokens becomes
 * g = min(text_len, n) groups with boundaries first + floor(j n / g).
 * Errors: VZ_ERR_INVALID for null pointers, n_seg < 0, t_total_ms <= 0,
 * L_a < 0 or L_a * t_total_ms beyond int64.
 */
VZ_API int voxzip_build_span_offsets(const int64_t *t_start_ms, const int64_t *t_end_ms,
                                     const float *conf, const int32_t *text_len, int32_t n_seg,
                                     int64_t t_total_ms, int32_t L_a, float conf_threshold,
                                     int32_t *off_out, int32_t *n_spans_out);

/*
 * Stage-1 semantic-anchored fusion (Sec. 3.2.1, Eq. 4 group average pooling,
 * the additive text anchor that follows it, and the chronological
 * concatenation of Eq. 5), applied to each layer's K and V per KV head.
 *
 *   k_out[l][h][j][:] = mean(k_in[l][h][span_off[j] .. span_off[j+1]-1][:])
 *                       (+ anchor_k[l][h][j][:] when anchor_k is not NULL)
 *   and the same for v; pos_out[l][j] = j; score_out[l][j] = 0
 *   for every layer l, KV head h and span j < n_spans.
 *
 *  k_in, v_in   [n_layers][kv_heads][T_in][d]  input (prefill) K and V.
 *               v_in and v_out may both be NULL: then only k is fused (and
 *               anchor_v must be NULL).  That serves the embedding-space form
 *               of Sec. 3.2.1 -- the audio-token input embeddings as k_in with
 *               n_layers = kv_heads = 1 and d = d_model, the text-token
 *               embeddings of each span as anchor_k (zero rows for
 *               background spans).
 *  d            64 or 128 for every dtype; fusion also takes any multiple of
 *               16 bytes (8 bf16 or 4 float32 elements) up to 16384.
 *  span_off     int32 [n_spans + 1], device.  Groups are contiguous and in
 *               time order: span_off[0] = 0, strictly increasing,
 *               span_off[n_spans] = T_in.  A background token is a span of
 *               length 1 (and is copied bit for bit).  Offsets are not read on
 *               the host; the kernel clamps them into [0, T_in], so malformed
 *               offsets give unspecified rows but never an out-of-range access.
 *  anchor_k/v   NULL, or [n_layers][kv_heads][n_spans][d] rows added after the mean.
 *  k_out, v_out [n_layers][kv_heads][cap_out][d]; slots >= n_spans untouched.
 *  score_out    float32 [n_layers][cap_out]; pos_out int32 [n_layers][cap_out].
 * Arithmetic: float32 sum in row order, IEEE division by the span length,
 * float32 anchor add, one rounding to dtype (nearest-even).
 * Errors: VZ_ERR_INVALID for null pointers (other than v_in/v_out together),
 * k_in/v_in aliasing an output or anchor_v without v_in; VZ_ERR_CAPACITY if
 * n_spans > cap_out; VZ_ERR_SHAPE if n_spans > T_in; VZ_ERR_UNSUPPORTED for
 * a row size fusion does not take.
 */
VZ_API int voxzip_fuse_spans(const void *k_in, const void *v_in, int32_t T_in,
                      const int32_t *span_off, int32_t n_spans,
                      const void *anchor_k, const void *anchor_v,
                      void *k_out, void *v_out, float *score_out, int32_t *pos_out,
                      int32_t n_layers, int32_t kv_heads, int32_t d, int32_t cap_out,
                      int32_t dtype, void *stream);

/*
 * One decode step for every layer: Sec. 3.1 Eq. 1 (append), Eq. 2 (attention)
 * and Sec. 3.2.2 Eq. 6 (temporally decayed accumulated score).
 *
 *  1. Append: k_cache/v_cache[l][g][len] = k_new/v_new[l][g];
 *     pos[l][len] = next_pos; the new slot's previous score is 0.
 *  2. Attend over slots 0..len (T = len + 1 keys): query head h reads KV head
 *     g = h / (n_q_heads / kv_heads);
 *       p[l][h][j] = softmax_j(sm_scale * q[l][h] . K[l][g][j]),
 *       out[l][h]  = sum_j p[l][h][j] * V[l][g][j].
 *  3. Score: score[l][j] = gamma * score[l][j] + sum_h p[l][h][j]  (j <= len).
 *
 *  q, out       [n_layers][n_q_heads][d];  k_new, v_new [n_layers][kv_heads][d].
 *  k_cache, v_cache, score, pos   in/out; slot len must exist (len + 1 <= cap).
 *  gamma        decay in [0, 1] (1 = plain accumulation).
 *  sm_scale     softmax scale; <= 0 selects 1 / sqrt(d).
 *  workspace    device scratch of at least voxzip_workspace_bytes(VZ_OP_DECODE,
 *               ...) bytes (per-chunk partial results), 16-byte aligned (as
 *               every workspace of this library); it needs no
 *               initialisation.  One workspace must not be used by two calls
 *               that can run at the same time.
 * The caller advances len and next_pos by one after the call.
 * Errors: VZ_ERR_INVALID (null pointer, gamma outside [0,1], len < 0),
 * VZ_ERR_CAPACITY (len + 1 > cap), VZ_ERR_SHAPE, VZ_ERR_UNSUPPORTED,
 * VZ_ERR_WORKSPACE.
 */
VZ_API int voxzip_decode_attend_score(const void *q, const void *k_new, const void *v_new,
                               void *k_cache, void *v_cache, float *score, int32_t *pos,
                               void *out, int32_t len, int32_t next_pos,
                               float gamma, float sm_scale,
                               int32_t n_layers, int32_t n_q_heads, int32_t kv_heads,
                               int32_t d, int32_t cap, int32_t dtype,
                               void *workspace, size_t ws_bytes, void *stream);

/*
 * Stage-2 eviction with in-place compaction (Sec. 3.2.2, Eq. 7-9).
 *
 * If len <= budget nothing moves.  Otherwise, per layer, with
 * M = n_recent (or budget / 5 when n_recent < 0) and T = n_sink:
 *   sinks   = slots with pos < T,
 *   recent  = slots with pos >= next_pos - M,
 *   middle  = the other slots;
 *   keep the N = budget - |sinks| - |recent| middle slots with the largest
 *   score (equal scores: the smaller position is kept), together with every
 *   sink and recent slot.  The kept rows of K, V, score and pos end up in slots
 *   0 .. budget-1 (kept rows already below `budget` do not move; kept rows above
 *   it fill the freed slots), so the resident set equals the concatenation of
 *   Eq. 7-8 up to slot order.
 *  next_pos     one past the newest position (positions must be < next_pos).
 *  kept_pos_out NULL, or int32 [n_layers][budget]: kept positions, ascending
 *               (filled also when nothing is evicted; needs next_pos <= 2^18).
 *  new_len_out  [host] receives min(len, budget).
 *  workspace    at least voxzip_workspace_bytes(VZ_OP_EVICT, ...) bytes.
 * Scores must be finite; -0 ranks as +0.
 * Errors: VZ_ERR_INVALID (null pointer, budget < 1, n_sink < 0,
 * n_sink + M > budget), VZ_ERR_CAPACITY (len > cap), VZ_ERR_SHAPE,
 * VZ_ERR_UNSUPPORTED, VZ_ERR_WORKSPACE.
 */
VZ_API int voxzip_evict_compact(void *k_cache, void *v_cache, float *score, int32_t *pos,
                         int32_t len, int32_t budget, int32_t n_sink, int32_t n_recent,
                         int32_t next_pos, int32_t *kept_pos_out, int32_t *new_len_out,
                         int32_t n_layers, int32_t kv_heads, int32_t d, int32_t cap,
                         int32_t dtype, void *workspace, size_t ws_bytes, void *stream);

/*
 * One generation step: Sec. 3.1 Eq. 1-2 and Sec. 3.2.2 Eq. 6 (the decode step
 * of voxzip_decode_attend_score at len, next_pos), then Sec. 3.2.2 Eq. 7-9
 * (voxzip_evict_compact of the len + 1 slots the step leaves, with next_pos +
 * 1), in one call.  The results are those of the two calls in that order, bit
 * for bit.  On the whole-range decode path (bf16, d = 128, at most 4 KV heads,
 * at least 128 (layer, KV head) pairs, len + 1 <= 8224, at most 256 moved
 * rows) the score fold and the selection run in one kernel, which takes the
 * new scores into the selection without re-reading them.
 *
 *  q ... sm_scale      as for voxzip_decode_attend_score.
 *  budget, n_sink, n_recent, kept_pos_out  as for voxzip_evict_compact; the
 *               eviction happens when len + 1 > budget (kept_pos_out is filled
 *               either way when given).
 *  new_len_out  [host] receives min(len + 1, budget); the caller's next len.
 *               The caller's next next_pos is next_pos + 1.
 *  workspace    at least voxzip_workspace_bytes(VZ_OP_DECODE_EVICT, ...) bytes;
 *               no initialisation needed; not shared by concurrent calls.
 * Errors: those of the two entry points.
 */
VZ_API int voxzip_decode_evict(const void *q, const void *k_new, const void *v_new,
                               void *k_cache, void *v_cache, float *score, int32_t *pos,
                               void *out, int32_t len, int32_t next_pos, float gamma,
                               float sm_scale, int32_t budget, int32_t n_sink,
                               int32_t n_recent, int32_t *kept_pos_out, int32_t *new_len_out,
                               int32_t n_layers, int32_t n_q_heads, int32_t kv_heads,
                               int32_t d, int32_t cap, int32_t dtype, void *workspace,
                               size_t ws_bytes, void *stream);

/*
 * The generation step of voxzip_decode_evict for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same arguments except the workspace,
 * the same launches and results, bit for bit.  Instead of a workspace it uses
 * a scratch array of VZ_NOALLOC_SCRATCH_BYTES that the library holds on each
 * GPU it runs on, from the first call on that GPU until the process ends.  It
 * allocates nothing and calls no allocating routine.
 *
 *  The call runs on the current device; `stream` must belong to it.
 *  Every call on one GPU shares that GPU's scratch array: calls that may
 *  overlap on one GPU (concurrent streams, threads) race and must be
 *  serialised by the caller.  The array needs no initialisation and may hold
 *  any earlier call's contents.
 *  Limit: calls whose workspace (voxzip_workspace_bytes(VZ_OP_DECODE_EVICT,
 *  ...)) exceeds VZ_NOALLOC_SCRATCH_BYTES return VZ_ERR_WORKSPACE with the
 *  sizes in voxzip_last_error() and queue nothing; the 48-layer, 4-KV-head,
 *  d = 128 cache of 8194 slots needs 52.5 MB.
 * Errors: those of voxzip_decode_evict, and VZ_ERR_HIP when the scratch
 * array's device address cannot be found.
 */
#define VZ_NOALLOC_SCRATCH_BYTES (64u << 20)
VZ_API int voxzip_decode_evict_noalloc(const void *q, const void *k_new, const void *v_new,
                                       void *k_cache, void *v_cache, float *score, int32_t *pos,
                                       void *out, int32_t len, int32_t next_pos, float gamma,
                                       float sm_scale, int32_t budget, int32_t n_sink,
                                       int32_t n_recent, int32_t *kept_pos_out,
                                       int32_t *new_len_out, int32_t n_layers, int32_t n_q_heads,
                                       int32_t kv_heads, int32_t d, int32_t cap, int32_t dtype,
                                       void *stream);

/*
 * Workspace bytes an operation needs for the given sizes (0 on a bad op).
 * n_q_heads is ignored for VZ_OP_EVICT.
 */
VZ_API size_t voxzip_workspace_bytes(int32_t op, int32_t n_layers, int32_t n_q_heads,
                              int32_t kv_heads, int32_t d, int32_t cap);

/*
 * Ragged batches
 * --------------
 * The *_ragged entry points serve n_seqs independent sequences (each with its
 * own length, capacity, budget and positions) in one launch sequence, so a
 * batch of sequences costs one call per step instead of one per sequence.
 * Every operation is the one of the single-sequence entry point, applied to
 * each sequence on its own (Sec. 3.2.1 per request, Sec. 3.1 and 3.2.2 per
 * decode step).
 *
 *  Packed layout: one cache [n_layers][kv_heads][total][d] (scores and
 *  positions [n_layers][total]); sequence s owns slots seq_base[s] ..
 *  seq_base[s] + cap[s] - 1 of every plane, and its slot j is the single-call
 *  slot j.  Sequences must not overlap.  total <= 2^26, 1 <= n_seqs <= 32768.
 *  Per-sequence values (seq_base int64, cap / len / budget / next_pos int32,
 *  [n_seqs] each) are DEVICE arrays, read by the kernels: host code never
 *  waits for them, so a whole serving loop can stay on the device.
 *  Idle batch slots: a sequence with cap[s] == 0 is an idle slot of the
 *  batch (no request holds it): every ragged call skips it without reading
 *  or writing anything of it and reports VZ_IDLE.  A serving loop retires a
 *  finished request by setting its cap to 0 and admits a new one into the
 *  slot by restoring the cap and fusing the request's prefill there, with no
 *  change to the launch shapes (a captured HIP graph of the step stays valid).
 *  status: NULL or int32 [n_seqs], device: receives VZ_OK per served
 *  sequence, VZ_IDLE per idle slot, or the error code of a sequence whose
 *  values are out of range; such a sequence is skipped (nothing of it is
 *  read or written, its outputs keep their previous contents).  Host-side
 *  errors are returned as usual.
 *
 * Workspace bytes of a ragged call (0 on a bad op or sizes out of range).
 */
VZ_API size_t voxzip_workspace_bytes_ragged(int32_t op, int32_t n_layers, int32_t n_q_heads,
                                            int32_t kv_heads, int32_t d, int64_t total,
                                            int32_t n_seqs);

/*
 * Ragged twin of voxzip_fuse_spans (Sec. 3.2.1, Eq. 4-5).
 *  k_in, v_in   [n_layers][kv_heads][total_in][d]; sequence s reads input rows
 *               in_base[s] .. in_base[s] + T_in[s] - 1 (int64 / int32 [n_seqs]).
 *  span_off     int32 [total_off]; sequence s's offsets are
 *               span_off[off_base[s] .. off_base[s] + n_spans[s]] (int64 /
 *               int32 [n_seqs]), relative to its first input row, with the
 *               rules of voxzip_fuse_spans.
 *  max_spans    host bound on every n_spans[s] (sizes the grid); a sequence
 *               with more spans gets VZ_ERR_CAPACITY.
 *  anchor_k/v   NULL, or laid out like the outputs (row j of sequence s at
 *               slot seq_base[s] + j).
 *  v_in, v_out, d  as for voxzip_fuse_spans: v_in and v_out both NULL fuse k
 *               alone; wide rows (the embedding-space form) are taken.
 *  k_out, v_out, score_out, pos_out  packed outputs; sequence s gets
 *               n_spans[s] rows from slot seq_base[s] (n_spans[s] <= cap[s]),
 *               pos = 0 .. n_spans[s] - 1, score 0.
 * Per-sequence errors (status): VZ_ERR_INVALID (a range outside its array),
 * VZ_ERR_SHAPE (n_spans > T_in), VZ_ERR_CAPACITY (n_spans > cap or > max_spans).
 * Returned errors: VZ_ERR_INVALID (null pointer, aliasing), VZ_ERR_SHAPE,
 * VZ_ERR_UNSUPPORTED.
 */
VZ_API int voxzip_fuse_spans_ragged(const void *k_in, const void *v_in, const int64_t *in_base,
                                    const int32_t *T_in, int64_t total_in, const int32_t *span_off,
                                    const int64_t *off_base, const int32_t *n_spans,
                                    int64_t total_off, int32_t max_spans, const void *anchor_k,
                                    const void *anchor_v, void *k_out, void *v_out, float *score_out,
                                    int32_t *pos_out, const int64_t *seq_base, const int32_t *cap,
                                    int64_t total, int32_t n_seqs, int32_t *status,
                                    int32_t n_layers, int32_t kv_heads, int32_t d, int32_t dtype,
                                    void *stream);

/*
 * Ragged twin of voxzip_decode_attend_score (Sec. 3.1 Eq. 1-2, Sec. 3.2.2
 * Eq. 6): every sequence s appends its token at slot len[s] with position
 * next_pos[s], attends over its len[s] + 1 slots and folds its scores.
 *  q, out       [n_seqs][n_layers][n_q_heads][d];
 *  k_new, v_new [n_seqs][n_layers][kv_heads][d].
 *  len, next_pos, cap, seq_base   device [n_seqs] (len and next_pos are not
 *               modified: the caller advances them, e.g. with one add).
 *  workspace    at least voxzip_workspace_bytes_ragged(VZ_OP_DECODE, ...)
 *               bytes; no initialisation needed; one call at a time per
 *               workspace.
 * Each sequence's results are bit-identical to a single-sequence call on
 * the same data.
 * Per-sequence errors (status): VZ_ERR_INVALID (negative len or next_pos, a
 * range outside the planes), VZ_ERR_CAPACITY (len + 1 > cap, or sequences that
 * overlap in the planes so that their work exceeds the bound the planes set).
 * Returned errors: as voxzip_decode_attend_score, plus VZ_ERR_SHAPE for
 * n_seqs or total out of range.
 */
VZ_API int voxzip_decode_attend_score_ragged(const void *q, const void *k_new, const void *v_new,
                                             void *k_cache, void *v_cache, float *score,
                                             int32_t *pos, void *out, const int64_t *seq_base,
                                             const int32_t *cap, const int32_t *len,
                                             const int32_t *next_pos, int64_t total,
                                             int32_t n_seqs, float gamma, float sm_scale,
                                             int32_t n_layers, int32_t n_q_heads, int32_t kv_heads,
                                             int32_t d, int32_t dtype, int32_t *status,
                                             void *workspace, size_t ws_bytes, void *stream);

/*
 * Ragged twin of voxzip_evict_compact (Sec. 3.2.2, Eq. 7-9): each sequence
 * with len[s] > budget[s] keeps its sinks (pos < n_sink), its recent window
 * (pos >= next_pos[s] - M, M = n_recent, or budget[s] / 5 when n_recent < 0)
 * and the top middle slots by score, compacted into its slots 0 ..
 * budget[s] - 1.
 *  kept_pos_out NULL, or int32 [n_layers][total]: sequence s's kept positions,
 *               ascending, from slot seq_base[s] (needs next_pos[s] <= 2^18).
 *  new_len_out  NULL, or device int32 [n_seqs]: min(len, budget) per served
 *               sequence (len for a skipped one); must not overlap len.
 *  workspace    at least voxzip_workspace_bytes_ragged(VZ_OP_EVICT, ...) bytes.
 * Per-sequence errors (status): VZ_ERR_INVALID (a range outside the planes,
 * budget < 1, n_sink + M > budget, next_pos < len), VZ_ERR_CAPACITY
 * (len > cap), VZ_ERR_UNSUPPORTED (kept_pos_out with next_pos > 2^18).
 * Returned errors: VZ_ERR_INVALID (null pointer, n_sink < 0, new_len_out
 * overlapping len), VZ_ERR_SHAPE, VZ_ERR_UNSUPPORTED, VZ_ERR_WORKSPACE.
 */
VZ_API int voxzip_evict_compact_ragged(void *k_cache, void *v_cache, float *score, int32_t *pos,
                                       const int64_t *seq_base, const int32_t *cap,
                                       const int32_t *len, const int32_t *budget,
                                       const int32_t *next_pos, int64_t total, int32_t n_seqs,
                                       int32_t n_sink, int32_t n_recent, int32_t *kept_pos_out,
                                       int32_t *new_len_out, int32_t *status, int32_t n_layers,
                                       int32_t kv_heads, int32_t d, int32_t dtype, void *workspace,
                                       size_t ws_bytes, void *stream);

/* Text of a status code (static storage). */
VZ_API const char *voxzip_status_string(int status);

/* Text of the last error raised on the calling thread ("" if none). */
VZ_API const char *voxzip_last_error(void);

/* ABI version, major * 100 + minor. */
VZ_API int voxzip_version(void);

#ifdef __cplusplus
}
#endif

#endif /* VOXZIP_H */
