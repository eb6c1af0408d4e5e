/*
 * atf.h -- C ABI of libatf.so: per-RoPE-wavelength windowed causal attention
 * (ATFlash, arXiv 2608.02947) on one AMD MI355X (gfx950).
 *
 * The method.  Queries and keys arrive already RoPE-rotated (q~, k~ of Sec. 3.1)
 * in the rotate-half layout: rotary pair r (r = 0 .. d/2-1, r = 0 the highest
 * frequency) is made of dims r and r + d/2.  The rotated score of a query at
 * position n and a key at position m splits exactly into one term per pair
 * (Sec. 3.1, eq:pair).  With theta_r = B^(-2r/d) (or an effective theta'_r when
 * the model scales its RoPE, Sec. 3.2 last paragraph), wavelength
 * lambda_r = 2*pi/theta_r (eq:lambda) and window w_r = min(k*lambda_r, N)
 * (Sec. 3.2, eq:window), the term of pair r is kept at distance z = n - m only
 * when z <= w_r.  Kept terms are summed and scaled; softmax and the product with
 * V are ordinary causal attention (FlashAttention recurrences, Fig. fa).  No token
 * is dropped: a cell whose every pair is pruned has score 0.
 *
 * Positions.  Query row i of a prefill call sits at position q_pos0 + i; key j
 * sits at position j.  Row i attends keys j <= q_pos0 + i (causal).  Because z
 * never exceeds the largest position, the min(., N) of eq:window never binds and
 * the integer threshold W_r = floor(k*lambda_r) decides: keep iff z <= W_r.
 *
 * Conventions shared by every entry point:
 *   - Return value: ATF_OK (0) or a negative ATF_E* code.  On error nothing is
 *     launched and no output is written; atf_last_error() describes the cause.
 *   - Device pointers are caller-owned, on the current HIP device, contiguous,
 *     and 16-byte aligned (lse: 4-byte aligned).  The library allocates no
 *     device memory.
 *   - ATF_OK from a call that launches work means "enqueued on hip_stream"
 *     (a hipStream_t; NULL = the null stream).  Faults surface at the caller's
 *     next synchronisation.  Launch failures return ATF_EHIP.
 *   - No C++ exception crosses this interface.  The library keeps no mutable
 *     global state besides a thread-local error string.
 *   - bf16 is IEEE binary32 truncated to its top 16 bits (stored as uint16);
 *     scores, softmax statistics and accumulators are fp32.
 */
#ifndef ATF_H
#define ATF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ATF_OK = 0,
    ATF_EINVAL = -1,       /* an argument is out of range, NULL, or misaligned */
    ATF_EUNSUPPORTED = -2, /* valid but not built: head_dim other than 64/128, GQA ratio > 8 not dividing */
    ATF_EWORKSPACE = -3,   /* decode workspace missing or smaller than atf_decode_workspace_bytes() */
    ATF_EHIP = -4          /* a HIP runtime call failed (launch error) */
};

/* Window parameters (Sec. 3.2: k is the only free parameter; the table follows
 * from the model's RoPE constants, or from its effective frequencies).
 *
 * With family != 0 the window is the member of the family of App. A (eq:family)
 *     w_r = min(max(k_r * lambda_r^gamma + a * (r + 1) / (d/2), beta), cap)
 * with k_r = k_profile[r] (or k for every pair when k_profile is NULL).  The
 * default window is k_r = k, gamma = 1, a = 0, beta = 0, cap = +INFINITY, and
 * family == 0 selects it whatever k_profile, gamma, a, beta and cap hold.  A
 * zero-initialised tail (family == 0, slice_pairs == 0) is the exact default window.
 * Examples: the variable-k profile (atf_retention_profile, 16 -> 2); uniform
 * k = 64; a ceiling cN (cap = c * N); the sliding window of width S (k_r = 0,
 * beta = cap = S); the linear window (k_r = 0, a = W). */
typedef struct atf_window {
    int32_t head_dim;        /* d; 64 or 128 for the GPU entry points, any even d >= 2 for the host ones */
    double rope_base;        /* B > 1; used only when inv_freq is NULL */
    double k;                /* retained periods, > 0 (>= 0 with family != 0); +INFINITY turns
                                the window off */
    const double *inv_freq;  /* optional HOST array [d/2] of effective theta'_r >= 0
                                (e.g. llama3 rope_scaling); NULL => theta_r = B^(-2r/d).
                                theta'_r == 0 is a position-free pair (never pruned, in the
                                family too: App. A treats it as a knob of its own). */
    int32_t family;          /* 0: default window; else eq:family with the fields below */
    const double *k_profile; /* optional HOST array [d/2] of k_r >= 0 (+INFINITY allowed);
                                NULL => k for every pair */
    double gamma;            /* wavelength exponent, finite */
    double a;                /* additive width in tokens (times (r+1)/(d/2)), finite, >= 0 */
    double beta;             /* floor in tokens, finite, >= 0 */
    double cap;              /* ceiling in tokens, >= 0; +INFINITY for none */
    int32_t slice_pairs;     /* 0 or 1: the exact window.  s > 1: the rounded slice of Sec. 3.3:
                                at each distance the kept pairs, a low-frequency slice, are
                                rounded up to a whole number of s-pair steps counted from the
                                lowest frequency (s = 8: 16-element MMA K-steps); needs a table
                                non-decreasing in r.  Read with family == 0 too. */
} atf_window;

/* Window table (Sec. 3.2 eq:window with eq:lambda, or App. A eq:family):
 * W_out[r] = floor(w_r) computed in fp64 and clamped to [0, 2^31 - 1] (the clamp is
 * exact because positions stay below 2^31 - 1, and w_r >= 0 always).  Pair r is kept
 * at distance z iff z <= W_out[r].  With slice_pairs = s > 1 the rounded slice keeps
 * pair r exactly where the window keeps the top pair of its s-pair step (steps counted
 * down from r = d/2 - 1), so W_out[r] is that pair's threshold.
 * W_out: host int32 array of d/2 entries.
 * Errors: ATF_EINVAL for a NULL pointer, odd or non-positive d, k <= 0 or NaN
 * (k < 0 with family), B <= 1 (without inv_freq), a negative/NaN inv_freq or
 * k_profile entry, a non-finite gamma, a or beta, a negative a, beta or cap, a
 * width that evaluates to NaN (0 * inf), slice_pairs < 0 or > d/2, or slice_pairs > 1
 * with a table that decreases somewhere in r. */
int atf_window_table(const atf_window *w, int32_t *W_out);

/* Retention profile k_r of App. A, r = 0 (highest frequency) .. d/2 - 1, into the
 * HOST array k_out[d/2]:
 *   ATF_PROFILE_CONSTANT    k_r = k_hi
 *   ATF_PROFILE_ARITHMETIC  k_r falls by (k_hi - k_lo)/(d/2 - 1) per pair, k_hi -> k_lo
 *                           (the variable-k profile: k_hi = 16, k_lo = 2)
 *   ATF_PROFILE_GEOMETRIC   k_r falls by the ratio (k_lo/k_hi)^(1/(d/2 - 1)) per pair
 * With one pair (d = 2) k_r = k_hi.  Errors: ATF_EINVAL for a NULL k_out, odd or
 * non-positive d, an unknown kind, k_hi or k_lo negative or not finite, or
 * (geometric) k_hi or k_lo == 0. */
enum { ATF_PROFILE_CONSTANT = 0, ATF_PROFILE_ARITHMETIC = 1, ATF_PROFILE_GEOMETRIC = 2 };
int atf_retention_profile(int32_t head_dim, int32_t kind, double k_hi, double k_lo,
                          double *k_out);

/* Retained inner-product terms of Sec. 4 for ONE (batch, query head): the number
 * of (causal cell, pair) terms kept by the window over query rows at positions
 * q_pos0 .. q_pos0 + n_q - 1 and keys 0 .. n_k - 1, and the number of causal
 * cells (the full-attention count is causal_cells * d/2).  Exact closed form per
 * pair; host only, no device work.  The reduction rate of Sec. 4 is
 * 1 - retained / (causal_cells * d/2).
 * Errors: ATF_EINVAL for NULL outputs, n_q < 0, q_pos0 < 0, n_k < 0, or a bad window. */
int atf_count_terms(const atf_window *w, int64_t n_q, int64_t q_pos0, int64_t n_k,
                    uint64_t *retained, uint64_t *causal_cells);

/* Prefill (chunked or whole): windowed causal attention of n_q query rows
 * against n_k keys, tiled with an online softmax; the window is applied as a
 * per-tile slice of the QK contraction axis (Sec. 3.3): fully kept pair-chunks
 * are MFMA K-steps, fully pruned ones are neither loaded nor multiplied, and
 * pairs whose window ends inside the tile are masked per element.  Keys and
 * values are read from the caches decode reads (atf_pack_kcache, atf_pack_vcache,
 * atf_cache_append), so one pair of caches serves a chunked prefill and the decode
 * steps after it, and a pruned chunk of a key is never read from HBM.
 *   q        bf16 [batch][n_q][h_q][d]        rotated queries            (device, read)
 *   k_cache  bf16 [batch][h_kv][d/16][cache_tokens][16]  rotated keys, pair-chunk-major,
 *            see atf_pack_kcache; keys 0 .. n_k - 1 are read          (device, read)
 *   v_cache  bf16 [batch][h_kv][ceil(cache_tokens/16)][d][16]  values in 16-token blocks,
 *            see atf_pack_vcache; tokens 0 .. n_k - 1 are used (later slots may hold
 *            anything)                                                (device, read)
 *   o        bf16 [batch][n_q][h_q][d]        output, O/l rounded to nearest even (device, written)
 *   lse      fp32 [batch][h_q][n_q]           natural-log sum of exp of the scaled scores (device, written)
 * cache_tokens is the number of tokens each batch entry of the caches is
 * allocated for (0 means n_k); a chunk of a longer prefill passes the positions of
 * its rows (q_pos0) and the keys written so far (n_k) against the same caches.
 * Query head h uses key/value head h / (h_q / h_kv).  softmax_scale <= 0 selects
 * 1/sqrt(d).  n_q == 0 is a no-op.
 * Errors: ATF_EINVAL (NULL/misaligned pointer, batch < 1, n_q < 0, n_k < 1,
 * q_pos0 < 0, q_pos0 + n_q > 2^31 - 1, n_k > 2^31 - 1, cache_tokens < n_k (when
 * non-zero) or > 2^31 - 1, h_q % h_kv != 0, bad window, non-finite scale);
 * ATF_EUNSUPPORTED (d not 64 or 128, or h_q / h_kv above 128 at d = 64 or above 256 at
 * d = 128: the query heads of one KV head share a workgroup's rows); ATF_EHIP. */
int atf_prefill(const void *q, const void *k_cache, const void *v_cache, void *o, float *lse,
                int32_t batch, int64_t n_q, int64_t n_k, int64_t q_pos0,
                int32_t h_q, int32_t h_kv, int64_t cache_tokens, const atf_window *w,
                float softmax_scale, void *hip_stream);

/* Pair-chunk width C_p (rotary pairs per chunk) of the decode K cache.  One
 * chunk of one token is 2*C_p bf16: dims [c*C_p, c*C_p + C_p) followed by dims
 * [d/2 + c*C_p, d/2 + c*C_p + C_p).  Returns 0 for an unsupported head_dim. */
int32_t atf_kcache_chunk_pairs(int32_t head_dim);

/* Repack a key cache from [batch][n_k][h_kv][d] (bf16, as prefill reads it) to
 * the pair-chunk-major decode layout [batch][h_kv][d/(2*C_p)][n_k][2*C_p], in
 * which every pair-chunk of a head is a contiguous stream over tokens, so that
 * decode reads only the tokens whose window still covers that chunk.  Pure data
 * movement (bit-exact).  k_bshd and k_pcm must not overlap.
 * Errors: ATF_EINVAL, ATF_EUNSUPPORTED (d), ATF_EHIP. */
int atf_pack_kcache(const void *k_bshd, void *k_pcm, int32_t batch, int64_t n_k,
                    int32_t h_kv, int32_t head_dim, void *hip_stream);

/* Rotate a whole unrotated K cache in one pass (RoPE at write time, the alternative
 * to rotating at read time of App. B): key t of every (batch, kv head) is turned to
 * position t, rotate-half convention of Sec. 2, in fp32 from the bf16 input and
 * rounded to bf16, and written to a second cache of the same layout, which
 * atf_prefill and atf_decode read as a pre-rotated cache.  Every (key, pair) is
 * rotated, whatever a window later keeps; the cost is one read and one write of the
 * cache and the rotated copy's memory.  Angles as in atf_prefill_unrotated (the
 * fixed-point fraction, exact for any position), evaluated directly per (key, pair).
 *   k_pcm  bf16 [batch][h_kv][d/16][cache_tokens][16], unrotated  (device, read)
 *   k_rot  bf16, same layout; keys 0 .. n_k - 1 written, later slots untouched
 *          (device, written; either k_pcm itself, which rotates the cache in place,
 *          or a buffer that does not overlap it)
 *   w      the window whose head_dim, and whose frequencies unless rope_inv_freq
 *          is given, define the rotation (its thresholds are not used)
 *   rope_inv_freq  host double [d/2] of theta_r, or NULL (as atf_prefill_unrotated)
 * cache_tokens 0 means n_k.
 * Errors: ATF_EINVAL (NULL/misaligned/partly overlapping buffers, batch < 1, n_k < 1,
 * h_kv < 1, n_k or cache_tokens >= 2^31 - 1, cache_tokens < n_k, a rotation frequency
 * that is negative, infinite or NaN); ATF_EUNSUPPORTED (d not 64 or 128, or
 * batch * h_kv * d/16 above 65535); ATF_EHIP. */
int atf_rotate_kcache(const void *k_pcm, void *k_rot, int32_t batch, int64_t n_k, int32_t h_kv,
                      int64_t cache_tokens, const atf_window *w, const double *rope_inv_freq,
                      void *hip_stream);

/* Bytes of the packed decode V cache for these sizes:
 * batch * h_kv * ceil(n_k / 16) * 16 * head_dim * 2.  Returns 0 for invalid sizes. */
size_t atf_vcache_bytes(int32_t batch, int64_t n_k, int32_t h_kv, int32_t head_dim);

/* Repack a value cache from [batch][n_k][h_kv][d] (bf16) to the decode layout
 * [batch][h_kv][ceil(n_k/16)][d][16]: blocks of 16 tokens stored d-major, so that
 * one 16-byte load gives the 8 tokens one lane of the PV matrix instruction
 * multiplies.  Within a block, slot 8*h + e of a d-row holds token
 * 8*(e/4) + 4*h + e%4 (h in {0,1}, e in 0..7), the token order of the score
 * fragments; tokens past n_k are zero.  Pure data movement (bit-exact).
 *   v_bshd  device, read;  v_pack  device, atf_vcache_bytes(...) bytes, written.
 * Both 16-byte aligned and not overlapping.
 * Errors: ATF_EINVAL, ATF_EUNSUPPORTED (d), ATF_EHIP. */
int atf_pack_vcache(const void *v_bshd, void *v_pack, int32_t batch, int64_t n_k,
                    int32_t h_kv, int32_t head_dim, void *hip_stream);

/* Append tokens to both caches: the keys and values of cache positions
 * pos0 .. pos0 + n_new - 1, given as the projections produce them, are written
 * into the pair-chunk-major K cache and the 16-token-block V cache of capacity
 * cache_tokens (layouts of atf_pack_kcache and atf_pack_vcache).  No other token's
 * data changes.  This is how a chunked prefill, an appended turn of a long session
 * (the interval prefill of App. C) or a decode step extends the caches that
 * atf_prefill and atf_decode read.  Pure data movement (bit-exact).
 *   k_new, v_new  bf16 [batch][n_new][h_kv][d]                   (device, read)
 *   k_cache       bf16 [batch][h_kv][d/16][cache_tokens][16]     (device, written at the new tokens)
 *   v_cache       bf16 [batch][h_kv][ceil(cache_tokens/16)][d][16] (device, written at the new tokens' slots)
 * All 16-byte aligned; the caches overlap neither each other nor the inputs.
 * n_new == 0 is a no-op.
 * Errors: ATF_EINVAL (NULL/misaligned/overlapping pointer, batch < 1, h_kv < 1,
 * n_new < 0, pos0 < 0, cache_tokens < 1 or > 2^31 - 1, pos0 + n_new > cache_tokens),
 * ATF_EUNSUPPORTED (d not 64 or 128), ATF_EHIP. */
int atf_cache_append(const void *k_new, const void *v_new, void *k_cache, void *v_cache,
                     int32_t batch, int64_t n_new, int64_t pos0, int32_t h_kv, int32_t head_dim,
                     int64_t cache_tokens, void *hip_stream);

/* atf_cache_append with RoPE on the way in: the new keys are given unrotated, as the
 * projections produce them, and key t is turned to its cache position pos0 + t
 * (rotate-half convention of Sec. 2, in fp32 from the bf16 input, rounded to bf16;
 * angles as in atf_rotate_kcache) while it is written into the pair-chunk-major cache:
 * the write-time rotation of App. B fused with the append, so the caches hold rotated
 * keys for atf_prefill and atf_decode.  Values as atf_cache_append.
 *   w              the window whose head_dim, and whose frequencies unless
 *                  rope_inv_freq is given, define the rotation (thresholds unused)
 *   rope_inv_freq  host double [d/2] of theta_r, or NULL (as atf_prefill_unrotated)
 * Everything else, errors included, as atf_cache_append, plus ATF_EINVAL for a NULL
 * window or a rotation frequency that is negative, infinite or NaN. */
int atf_cache_append_rotated(const void *k_new, const void *v_new, void *k_cache, void *v_cache,
                             int32_t batch, int64_t n_new, int64_t pos0, int32_t h_kv,
                             int64_t cache_tokens, const atf_window *w,
                             const double *rope_inv_freq, void *hip_stream);

/* Bytes of device workspace that atf_decode and atf_decode_ragged need for these
 * sizes (split-KV partial softmax states; the figure covers the split plans of both
 * calls).  Returns 0 for invalid sizes. */
size_t atf_decode_workspace_bytes(int32_t batch, int32_t h_q, int32_t h_kv, int64_t n_k,
                                  int32_t head_dim);

/* Decode: one query token per batch row at position q_pos, against keys
 * 0 .. min(q_pos, n_k - 1) of that row's cache (the last query row of Fig. fa).
 * The cache is split over tokens; each split keeps partial (max, normaliser,
 * output) states that a second kernel merges (split-KV, Sec. 5).  For pair-chunk
 * c only the token suffix whose distance is within the chunk's largest window
 * is read; pairs whose window ends inside that suffix are masked per token.
 *   q        bf16 [batch][h_q][d]                                   (device, read)
 *   k_cache  bf16 [batch][h_kv][d/16][cache_tokens][16] pair-chunk-major,
 *            see atf_pack_kcache                                     (device, read)
 *   v_cache  bf16 [batch][h_kv][ceil(cache_tokens/16)][d][16] packed 16-token
 *            blocks, see atf_pack_vcache                             (device, read)
 *   o        bf16 [batch][h_q][d]                                   (device, written)
 *   lse      fp32 [batch][h_q]                                      (device, written)
 *   workspace: device, >= atf_decode_workspace_bytes(batch, h_q, h_kv, n_k, d)
 *              bytes, 16-byte aligned, caller-owned; contents are scratch.
 * cache_tokens is the number of tokens each batch entry of the caches is
 * allocated for (0 means n_k); only tokens below n_k are read.
 * Errors: ATF_EINVAL (pointers, sizes, q_pos < 0, q_pos > 2^31 - 2, cache_tokens
 * < n_k when non-zero, bad window or scale), ATF_EUNSUPPORTED (d not 64/128),
 * ATF_EWORKSPACE, ATF_EHIP.
 * The query heads of one KV head are the columns of the matrix instructions
 * (up to 32 per workgroup; larger groups are split over workgroups by their
 * largest divisor <= 32).  Deterministic: equal inputs give equal bits. */
int atf_decode(const void *q, const void *k_cache, const void *v_cache, void *o, float *lse,
               int32_t batch, int64_t n_k, int64_t q_pos, int32_t h_q, int32_t h_kv,
               int64_t cache_tokens, const atf_window *w, float softmax_scale,
               void *workspace, size_t workspace_bytes, void *hip_stream);

/* Size in bytes of the library's own decode scratch array (atf_decode_noalloc). */
#define ATF_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/* atf_decode without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, allocation-free serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, layouts, window, kernels and
 * results as atf_decode, bit for bit; the split partial states go to a
 * file-scope device array of ATF_DECODE_NOALLOC_SCRATCH_BYTES (16 MiB) inside the
 * library instead of a caller workspace.  The call allocates nothing (no
 * hipMalloc, hipFree or allocating library routine); the first call on a device
 * resolves that device's copy of the array.
 * Limit: the partial states of these sizes, atf_decode_workspace_bytes(batch,
 * h_q, h_kv, n_k, head_dim) for the uniform plan (about batch * splits * h_q *
 * (4 head_dim + 8) bytes; 3.7 MB for 28 query heads / 4 KV heads, d = 128, at 1M
 * keys), must fit in the array, else ATF_EWORKSPACE and nothing is launched.
 * Sharing: every device holds its own copy for the life of the process, and all
 * calls on one device share it and leave their partial states in it, so two
 * calls that may run at the same time on one device (different streams, host
 * threads) race: serialise them.  Nothing needs to be cleared between calls.
 * Errors: as atf_decode (ATF_EWORKSPACE only for the limit above; ATF_EHIP also
 * when the array's address cannot be resolved). */
int atf_decode_noalloc(const void *q, const void *k_cache, const void *v_cache, void *o,
                       float *lse, int32_t batch, int64_t n_k, int64_t q_pos, int32_t h_q,
                       int32_t h_kv, int64_t cache_tokens, const atf_window *w,
                       float softmax_scale, void *hip_stream);

/* Decode of a ragged batch: row b holds one query token at position q_pos_rows[b]
 * against keys 0 .. min(q_pos_rows[b], n_k_rows[b] - 1) of its own cache entry
 * (Sec. 5: the last query row of each sequence, for a batch of sequences of
 * different lengths).  Everything else is atf_decode: same layouts, window,
 * split-KV partial states and merge.  The split plan follows the rows' lengths
 * on the device: the batch's causal keys are cut into spans of equal length (a
 * multiple of 128 tokens, about 2048 workgroups in all), each row into whole
 * spans of its own keys, so a short row takes few workgroups and a long one many.
 *   n_k_rows    int32 [batch], DEVICE, 4-byte aligned: keys of each row's cache
 *   q_pos_rows  int32 [batch], DEVICE, 4-byte aligned: query position of each row
 *   max_n_k     host bound on n_k_rows (1 .. cache_tokens); the workspace is
 *               atf_decode_workspace_bytes(batch, h_q, h_kv, max_n_k, d)
 * The row arrays stay on the device (no host synchronisation).  The kernel clamps
 * each row to n_k_rows[b] in [0, max_n_k] and q_pos_rows[b] in [0, 2^31 - 3], so it
 * never reads outside the row's cache whatever the arrays hold; values outside
 * those ranges are a caller error that this clamping makes harmless, not a
 * supported input.  A row with no key (n_k_rows[b] == 0) has an empty softmax:
 * its output is 0 and its LSE is -INFINITY.
 * Errors: as atf_decode, plus ATF_EINVAL for NULL/misaligned row arrays and
 * max_n_k < 1 or > cache_tokens.  Deterministic: equal inputs give equal bits. */
int atf_decode_ragged(const void *q, const void *k_cache, const void *v_cache, void *o, float *lse,
                      int32_t batch, const int32_t *n_k_rows, const int32_t *q_pos_rows,
                      int64_t max_n_k, int32_t h_q, int32_t h_kv, int64_t cache_tokens,
                      const atf_window *w, float softmax_scale, void *workspace,
                      size_t workspace_bytes, void *hip_stream);

/* Paged caches (a serving layout the paper does not use: its decode reads one
 * contiguous cache per request, Sec. 5; the window applies per 32-token block of a
 * page exactly as in atf_decode): the K and V caches of all rows live in pools of
 * pages of page_tokens tokens (a multiple of 32, the decode kernel's token block).
 * Page i of the pools holds
 *   k_pages  bf16 [num_pages][h_kv][d/16][page_tokens][16]  pair-chunk-major within
 *            the page (chunk c of a head is a contiguous stream over its tokens, as in
 *            the contiguous K cache: a pruned chunk is never read)
 *   v_pages  bf16 [num_pages][h_kv][page_tokens/16][d][16]   16-token blocks as in
 *            the contiguous V cache (see atf_pack_vcache)
 * Row b's token t lives in page block_table[b * max_pages_per_row + t / page_tokens],
 * at token t % page_tokens of that page.  block_table: int32, DEVICE.  Pages may be
 * shared between rows or unused; the library never allocates or frees them.
 *
 * Write n_new tokens of every row, at row positions pos0 .. pos0 + n_new - 1, into
 * the pages the block table names for them.  Pure data movement (bit-exact).
 *   k_new, v_new  bf16 [batch][n_new][h_kv][d]                   (device, read)
 * Page entries outside [0, num_pages) are skipped (the caller's error; nothing is
 * written outside the pools).  The slots of a page's 16-token V block that the call
 * does not write keep their contents.  n_new == 0 is a no-op.
 * Errors: ATF_EINVAL (NULL/misaligned pointer, batch < 1, h_kv < 1, n_new < 0, pos0 < 0,
 * page_tokens not a positive multiple of 32, num_pages < 1, max_pages_per_row < 1,
 * pos0 + n_new > max_pages_per_row * page_tokens), ATF_EUNSUPPORTED (d not 64/128),
 * ATF_EHIP. */
int atf_cache_append_paged(const void *k_new, const void *v_new, void *k_pages, void *v_pages,
                           const int32_t *block_table, int32_t max_pages_per_row,
                           int32_t num_pages, int32_t page_tokens, int32_t batch,
                           int64_t n_new, int64_t pos0, int32_t h_kv, int32_t head_dim,
                           void *hip_stream);

/* atf_cache_append_paged with RoPE on the way in: the new keys are given unrotated and
 * key t of row b is turned to its position pos0 + t as it is written into its page
 * (rotation as atf_cache_append_rotated).  Values, tables, pools, clamping of table
 * entries and errors as atf_cache_append_paged, plus ATF_EINVAL for a NULL window or a
 * rotation frequency that is negative, infinite or NaN.  The head dimension is the
 * window's. */
int atf_cache_append_paged_rotated(const void *k_new, const void *v_new, void *k_pages,
                                   void *v_pages, const int32_t *block_table,
                                   int32_t max_pages_per_row, int32_t num_pages,
                                   int32_t page_tokens, int32_t batch, int64_t n_new,
                                   int64_t pos0, int32_t h_kv, const atf_window *w,
                                   const double *rope_inv_freq, void *hip_stream);

/* Decode of a ragged batch over paged caches: atf_decode_ragged with row b's keys read
 * through its block table (layouts above).  max_n_k bounds n_k_rows and must not
 * exceed max_pages_per_row * page_tokens; the workspace is
 * atf_decode_workspace_bytes(batch, h_q, h_kv, max_n_k, d).  The kernel clamps row
 * lengths and positions as atf_decode_ragged does and page entries to
 * [0, num_pages), so it never reads outside the pools whatever the arrays hold;
 * such values are a caller error made harmless, not a supported input.
 * Errors: as atf_decode_ragged, plus ATF_EINVAL for a NULL/misaligned block table,
 * page_tokens not a positive multiple of 32, num_pages < 1, max_pages_per_row < 1,
 * max_n_k > max_pages_per_row * page_tokens.  Deterministic. */
int atf_decode_paged(const void *q, const void *k_pages, const void *v_pages, void *o, float *lse,
                     int32_t batch, const int32_t *block_table, int32_t max_pages_per_row,
                     int32_t num_pages, int32_t page_tokens, const int32_t *n_k_rows,
                     const int32_t *q_pos_rows, int64_t max_n_k, int32_t h_q, int32_t h_kv,
                     const atf_window *w, float softmax_scale, void *workspace,
                     size_t workspace_bytes, void *hip_stream);

/* Decode from UNROTATED caches: RoPE applied at read time (App. B, cache footprint
 * versus rotation count).  q and the K cache hold the vectors before rotation; the
 * kernel rotates the query to its position and each key to its position (key j at
 * position j of its row) as it reads it, so only the pairs the window keeps are ever
 * rotated: a pruned pair is neither read nor rotated.  Rotate-half convention of
 * Sec. 2 (pair r = dims r and r + d/2, angle position * theta_r), in fp32 from the
 * bf16 inputs, rounded to bf16 before the matrix products; the angle is exact for any
 * position (theta_r / (2 pi) held as a 0.64 fixed-point fraction).
 *   rope_inv_freq  host double [d/2] of the rotation's theta_r, or NULL: the window's
 *                  frequencies (w->inv_freq if set, else rope_base^(-2r/d))
 * Everything else is atf_decode (atf_decode_unrotated), atf_decode_ragged
 * (atf_decode_ragged_unrotated: row b's key t at position t) or atf_decode_paged
 * (atf_decode_paged_unrotated): same layouts, window, workspace, errors, plus
 * ATF_EINVAL for a rotation frequency that is negative, infinite or NaN.  V is never
 * rotated.  Deterministic: equal inputs give equal bits. */
/* Prefill from UNROTATED caches: RoPE applied at read time (App. B), as in
 * atf_decode_unrotated.  Query row i (position q_pos0 + i) is rotated once as the
 * workgroup loads it; each key j (position j) is rotated chunk by chunk after the chunk
 * lands in LDS, and only the pair-chunks the window keeps for the tile are loaded and
 * rotated, so a pruned pair of a key is neither read nor rotated.  Rotate-half
 * convention of Sec. 2 in fp32 from the bf16 inputs, rounded to bf16 before the matrix
 * products; the key's angle (block start + offset) * theta_r is formed by angle
 * addition from the block start's angle (0.64 fixed-point fraction, exact for any
 * position) and a table of the 32 offsets' angles, so it is within a few fp32 ulps of
 * the exact angle.
 *   rope_inv_freq  host double [d/2] of the rotation's theta_r, or NULL: the window's
 *                  frequencies (w->inv_freq if set, else rope_base^(-2r/d))
 * Everything else is atf_prefill: same layouts, window, errors, plus ATF_EINVAL for a
 * rotation frequency that is negative, infinite or NaN.  V is never rotated. */
int atf_prefill_unrotated(const void *q, const void *k_cache, const void *v_cache, void *o,
                          float *lse, int32_t batch, int64_t n_q, int64_t n_k, int64_t q_pos0,
                          int32_t h_q, int32_t h_kv, int64_t cache_tokens, const atf_window *w,
                          const double *rope_inv_freq, float softmax_scale, void *hip_stream);

int atf_decode_unrotated(const void *q, const void *k_cache, const void *v_cache, void *o,
                         float *lse, int32_t batch, int64_t n_k, int64_t q_pos, int32_t h_q,
                         int32_t h_kv, int64_t cache_tokens, const atf_window *w,
                         const double *rope_inv_freq, float softmax_scale, void *workspace,
                         size_t workspace_bytes, void *hip_stream);
int atf_decode_ragged_unrotated(const void *q, const void *k_cache, const void *v_cache, void *o,
                                float *lse, int32_t batch, const int32_t *n_k_rows,
                                const int32_t *q_pos_rows, int64_t max_n_k, int32_t h_q,
                                int32_t h_kv, int64_t cache_tokens, const atf_window *w,
                                const double *rope_inv_freq, float softmax_scale,
                                void *workspace, size_t workspace_bytes, void *hip_stream);
int atf_decode_paged_unrotated(const void *q, const void *k_pages, const void *v_pages, void *o,
                               float *lse, int32_t batch, const int32_t *block_table,
                               int32_t max_pages_per_row, int32_t num_pages, int32_t page_tokens,
                               const int32_t *n_k_rows, const int32_t *q_pos_rows,
                               int64_t max_n_k, int32_t h_q, int32_t h_kv, const atf_window *w,
                               const double *rope_inv_freq, float softmax_scale, void *workspace,
                               size_t workspace_bytes, void *hip_stream);

/* Message of the most recent failed call on this thread ("" if none). */
const char *atf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ATF_H */
