/*
 * hwkv.h -- C ABI of the HeadWiseKV grouped-cache runtime for MI355X (gfx950).
 *
 * HeadWiseKV gives every physical KV head (l, h) of a residual full-attention
 * layer -- a "unit" -- a static history: full, or a recent window of w_lh
 * tokens, chosen from a small codebook of window levels (paper: Method,
 * "Structured Residency Model", the policy matrix a_lh over
 * W = {w_1..w_K, full}).  The runtime stores that history as physical
 * residency, not as a mask over a full cache (Method, "From Policy to
 * Physical Residency"): storage is allocated per (window level, unit) before
 * prefill, each unit reads and writes only its own slice, and the query heads
 * of a GQA group read their shared KV-head slice; per-head outputs are
 * concatenated before gating and the output projection.
 *
 * Residency of a finite unit with window w and S sink tokens, for a sequence
 * of length n (positions 0..n-1):  R(n) = {p < S} U {p >= n - w}, of size
 * min(n, S + w).  The window follows the paper's J_t(w) (Method, sequential
 * calibration: positions t-w+1..t, the query's own token included); sinks
 * are an additive prefix as in the paper's sink+recent control (Appendix,
 * baseline controls: 4 sinks + 90,364 recent = a 90,368-token cache).
 * S = 0 is exactly the paper's suffix window.  A window with S + w >= max_ctx
 * is full ("any w >= C is equivalent to full").
 *
 * Physical slot of position p in its unit: p for full units and sinks,
 * S + ((p - S) mod w) otherwise (a ring).  After any sequence of calls the
 * occupied slots of a (unit, sequence) are exactly [0, min(n, cap)).
 *
 * Conventions for every entry point:
 *   - returns HWKV_OK (0) or one of the positive error codes below; on error no
 *     state changes and hwkv_last_error() describes the failure;
 *   - all validation happens on the host before any device work;
 *   - handles are opaque; hwkv_policy_set copies its arrays and
 *     hwkv_cache_alloc copies the policy (the policy may be freed after);
 *   - device pointers (k, v, q, out, workspace, dev_buf) are caller-owned
 *     device memory, 16-byte aligned, contiguous; the library never frees
 *     them.  bf16 tensors are passed as raw 16-bit bf16 storage;
 *   - `stream` is a borrowed hipStream_t passed as void* (NULL = the null
 *     stream); device work is enqueued on it asynchronously and launch errors
 *     are reported as HWKV_EDEVICE;
 *   - a cache is not thread-safe: calls on one cache must be serialised, and
 *     the host keeps the sequence lengths, so calls on one cache must be
 *     issued in the order the device should execute them.
 */
#ifndef HWKV_H
#define HWKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HWKV_OK 0
#define HWKV_EINVAL 1    /* invalid argument */
#define HWKV_ENOMEM 2    /* host or device memory, or a too-small buffer */
#define HWKV_ECAPACITY 3 /* a full unit would exceed max_ctx */
#define HWKV_ESTATE 4    /* call does not match the cache state */
#define HWKV_EDEVICE 5   /* HIP runtime or launch error */

/* Cache formats p_KV of the stored keys and values (Method, Eq.
 * nominal-storage: the format enters the storage through the effective bytes
 * per element b^K, b^V; a format that changes numerical execution is used by
 * every reader of the cache).  Inputs are always bf16; the cache stores:
 *   HWKV_KV_BF16      the bf16 input as is (2 bytes per element);
 *   HWKV_KV_F16       IEEE binary16 of the input, round to nearest even,
 *                     overflow to infinity (2 bytes);
 *   HWKV_KV_FP8_E4M3  OCP FP8 E4M3 ("E4M3FN": bias 7, subnormals m * 2^-9,
 *                     largest finite 448, no infinities, S.1111.111 = NaN) of
 *                     x / s, where s is the fp32 scale of the element's
 *                     (layer, KV head) and tensor (K or V): the quotient is the
 *                     correctly rounded fp32 division, rounded to nearest even
 *                     and saturated to +-448, NaN kept (1 byte).
 * The value an element contributes to attention is its stored value (times s
 * for fp8). */
#define HWKV_KV_BF16 0
#define HWKV_KV_F16 1
#define HWKV_KV_FP8_E4M3 2

typedef struct hwkv_policy hwkv_policy;
typedef struct hwkv_cache hwkv_cache;

/* Text of the last error raised on the calling thread ("" if none).  The
 * pointer stays valid until the next call on that thread. */
const char *hwkv_last_error(void);

/* ------------------------------------------------------------------------ */
/* Policy: the static layer x KV-head matrix over a window codebook         */
/* (Method, "Structured Residency Model"; Appendix, runtime realization:    */
/* the matrix is loaded once and never recomputed from the prompt).         */
/* ------------------------------------------------------------------------ */

/* Create a policy.
 *   n_layers, n_kv_heads  units are (layer, kv_head), layer-major;
 *                         1 <= n_kv_heads <= 64
 *   n_q_heads             multiple of n_kv_heads; query head q reads KV head
 *                         q / (n_q_heads / n_kv_heads) (contiguous GQA
 *                         groups); group size 1, 2, 4, 6 or 8
 *   head_dim              64, 128 or 256 (K and V share it)
 *   n_sinks               S >= 0, shared by all finite units
 *   n_levels              codebook size K + 1 (>= 1)
 *   level_window[k]       window of level k: > 0 finite, 0 = full history
 *   level_of_unit[u]      level index of unit u = layer * n_kv_heads + h
 * Units with the same level form one storage group (same capacity, disjoint
 * contents).  EINVAL on any out-of-range value. */
int hwkv_policy_set(hwkv_policy **out, int32_t n_layers, int32_t n_kv_heads,
                    int32_t n_q_heads, int32_t head_dim, int32_t n_sinks,
                    int32_t n_levels, const int64_t *level_window,
                    const int32_t *level_of_unit);

int hwkv_policy_free(hwkv_policy *policy);

/* Shape of a policy: layers, KV heads, query heads, head_dim, sink count and
 * codebook size (any output pointer may be NULL). */
int hwkv_policy_shape(const hwkv_policy *policy, int32_t *n_layers,
                      int32_t *n_kv_heads, int32_t *n_q_heads, int32_t *head_dim,
                      int32_t *n_sinks, int32_t *n_levels);


/* Nominal K/V bytes of the policy at context ctx (Eq. nominal-storage with
 * bf16 K and V: r_C(w) * head_dim * (2 + 2) per unit and sequence, where
 * r_C(w) = min(S + w, ctx) for a finite window and ctx for full). */
int hwkv_policy_bytes(const hwkv_policy *policy, int64_t ctx, double *bytes);

/* Eq. nominal-storage under cache format kv_format: r_C(w) * head_dim *
 * (b^K + b^V) per unit and sequence, with b = 2 (bf16, f16) or 1 (fp8). */
int hwkv_policy_bytes_format(const hwkv_policy *policy, int64_t ctx,
                             int32_t kv_format, double *bytes);

/* Normalized rate R_C (Eq. normalized-rate): nominal bytes divided by the
 * all-full policy's nominal bytes at the same ctx.  Host only. */
int hwkv_policy_rate(const hwkv_policy *policy, int64_t ctx, double *rate);

/* ------------------------------------------------------------------------ */
/* Cache: grouped physical storage allocated before prefill                  */
/* (Method, "From Policy to Physical Residency"; Appendix, physical cache    */
/* realization: per-(window, KV head) groups, disjoint per-layer contents).  */
/* ------------------------------------------------------------------------ */

/* Exact device bytes hwkv_cache_alloc needs for `batch` sequences of at most
 * max_ctx tokens: per unit and sequence, cap rounded up to a multiple of 64
 * token rows (the K tile), times head_dim * (2 + 2) bytes, where cap = max_ctx
 * for full units (or S + w >= max_ctx) and S + w otherwise.  Equals
 * batch x Eq. nominal-storage at ctx = max_ctx up to that rounding.
 * 1 <= max_ctx, and max_ctx (rounded up to 64) * head_dim * 2 < 2^31, the
 * bytes of one unit's K or V per sequence (4,194,240 tokens at head_dim 256).
 * EINVAL otherwise or on size_t overflow. */
int hwkv_cache_bytes(const hwkv_policy *policy, int32_t batch, int64_t max_ctx,
                     size_t *bytes);

/* hwkv_cache_bytes for a cache of format kv_format: element size b (2 or 1)
 * in place of 2, and the limit max_ctx (rounded up to 64) * head_dim * b <
 * 2^31.  EINVAL on an unknown format. */
int hwkv_cache_bytes_format(const hwkv_policy *policy, int32_t batch,
                            int64_t max_ctx, int32_t kv_format, size_t *bytes);

/* Allocate a cache.  dev_buf == NULL: the library allocates (hipMalloc on the
 * current device), zero-fills, and owns the memory.  Otherwise the caller's
 * device buffer of buf_bytes is adopted as is (ENOMEM if smaller than
 * hwkv_cache_bytes); it must stay valid until hwkv_cache_free.  Every
 * sequence length starts at 0. */
int hwkv_cache_alloc(hwkv_cache **out, const hwkv_policy *policy,
                     int32_t batch, int64_t max_ctx, void *dev_buf,
                     size_t buf_bytes);

/* hwkv_cache_alloc for a cache of format kv_format (hwkv_cache_alloc is the
 * bf16 case).  k_scale, v_scale: host fp32 [n_layers][n_kv_heads], the fp8
 * scales s of K and V per unit (copied; NULL = all 1.0); each must be
 * positive, finite and normal.  For the 16-bit formats they must be NULL.
 * Buffer size rules as for hwkv_cache_alloc with hwkv_cache_bytes_format.
 * EINVAL on an unknown format or a bad scale. */
int hwkv_cache_alloc_format(hwkv_cache **out, const hwkv_policy *policy,
                            int32_t batch, int64_t max_ctx, int32_t kv_format,
                            const float *k_scale, const float *v_scale,
                            void *dev_buf, size_t buf_bytes);

/* Format of a cache and, if the pointers are non-NULL, its scales (host fp32
 * [n_layers][n_kv_heads] each; all 1.0 for the 16-bit formats). */
int hwkv_cache_format(const hwkv_cache *cache, int32_t *kv_format,
                      float *k_scale, float *v_scale);

/* Paged storage of the full units, for ragged batches (the reservation of
 * max_ctx rows per full unit and sequence is what dominates a batch of short
 * and long sequences; the paper cites paged memory management as orthogonal
 * to its retention policy).  In a paged cache the finite units keep their
 * S + w rows per sequence; the full units hold no fixed storage and take
 * pages of HWKV_PAGE_TOKENS token rows (K and V of one unit and sequence)
 * from one pool as their sequences grow.  Calls that need pages take them
 * from the pool first and fail with ENOMEM, changing nothing, when it has
 * too few; hwkv_cache_reset_seq returns a sequence's pages.  Results are
 * those of an unpaged cache. */
#define HWKV_PAGE_TOKENS 256

/* Exact device bytes of a paged cache: the finite units as in
 * hwkv_cache_bytes_format, a pool of n_pages pages of
 * 2 * HWKV_PAGE_TOKENS * head_dim * b bytes, and the page table (4 bytes per
 * page of every full unit and sequence at max_ctx), each part 256-byte
 * aligned.  n_pages >= 0.  EINVAL as hwkv_cache_bytes_format. */
int hwkv_cache_bytes_paged(const hwkv_policy *policy, int32_t batch,
                           int64_t max_ctx, int32_t kv_format, int64_t n_pages,
                           size_t *bytes);

/* Allocate a paged cache: arguments as hwkv_cache_alloc_format, plus the pool
 * size n_pages (pages of HWKV_PAGE_TOKENS rows).  The pool starts free. */
int hwkv_cache_alloc_paged(hwkv_cache **out, const hwkv_policy *policy,
                           int32_t batch, int64_t max_ctx, int32_t kv_format,
                           const float *k_scale, const float *v_scale,
                           int64_t n_pages, void *dev_buf, size_t buf_bytes);

/* Pool size and free pages of a paged cache (0 and 0 for an unpaged one). */
int hwkv_cache_pages(const hwkv_cache *cache, int64_t *total,
                     int64_t *free_pages);

/* Release sequence `seq`: its length becomes 0 in every layer and the pages
 * of its full units return to the pool (host bookkeeping only: no device
 * work, ordered with the cache's other calls as they are issued).  Valid on
 * any cache; a released sequence is filled again from position 0. */
int hwkv_cache_reset_seq(hwkv_cache *cache, int32_t seq);

/* Release the cache; frees device memory only if the library allocated it.
 * The caller must make sure no enqueued work still uses the cache. */
int hwkv_cache_free(hwkv_cache *cache);

/* Host mirror of the length n of sequence `seq` in `layer`. */
int hwkv_cache_seq_len(const hwkv_cache *cache, int32_t layer, int32_t seq,
                       int64_t *n);

/* Capacity (token rows holding data, before tile rounding) of unit
 * (layer, kv_head) per sequence, and its window after canonicalisation
 * (0 = full). */
int hwkv_cache_unit_info(const hwkv_cache *cache, int32_t layer,
                         int32_t kv_head, int64_t *capacity, int64_t *window);

/* ------------------------------------------------------------------------ */
/* Data path                                                                 */
/* ------------------------------------------------------------------------ */

/* Prefill materialisation of tokens [pos0, pos0 + n_tokens) of sequence
 * `seq` in `layer`: only positions still retained once the sequence has
 * length pos0 + n_tokens are written, each into its slot; no full-length
 * cache is ever formed (Method, physical residency; Intro: storage shrinks
 * before the cache is built).  Then n(layer, seq) = pos0 + n_tokens.
 *   k, v   device bf16 [n_tokens][n_kv_heads][head_dim], post-RoPE keys,
 *          stored in the cache's format.
 * ESTATE if pos0 != n(layer, seq); ECAPACITY if a full unit would pass
 * max_ctx; ENOMEM if a paged cache's pool has too few pages; n_tokens == 0
 * is a no-op. */
int hwkv_prefill_write(hwkv_cache *cache, int32_t layer, int32_t seq,
                       int64_t pos0, int64_t n_tokens, const void *k,
                       const void *v, void *stream);

/* Prefill attention of tokens [pos0, pos0 + n_tokens) of sequence `seq` in
 * `layer`, before they are materialised: query token t (t in the chunk) of
 * query head qh attends over R(t + 1) restricted to [0, t] of KV head
 * qh / G -- positions s <= t with s < S or s >= t + 1 - w, every s <= t for a
 * full unit (Eqs. conditional-attention-weight and conditional-attention,
 * z = scale * q.k, with the sink prefix).  Keys below pos0 are read from the
 * cache in its current state; keys in [pos0, t] from k and v.  The cache is
 * not changed: follow with hwkv_prefill_write of the same chunk.
 *   q     device bf16 [n_tokens][n_q_heads][head_dim], post-RoPE
 *   k, v  device bf16 [n_tokens][n_kv_heads][head_dim], post-RoPE keys
 *   out   device fp32 [n_tokens][n_q_heads][head_dim] (pre-gate)
 * bf16 MFMA products with fp32 accumulation; the softmax weights enter the
 * value product rounded to bf16.  ESTATE if pos0 != n(layer, seq);
 * ECAPACITY if pos0 + n_tokens > max_ctx; EINVAL on bad indices, null
 * pointers, a non-finite or non-positive scale, or a cache whose format is
 * not bf16 (hwkv_prefill_attn_ws takes every format); n_tokens == 0 is a
 * no-op. */
int hwkv_prefill_attn(hwkv_cache *cache, int32_t layer, int32_t seq,
                      int64_t pos0, int64_t n_tokens, const void *q,
                      const void *k, const void *v, float scale, void *out,
                      void *stream);

/* Device workspace bytes hwkv_prefill_attn_ws needs on this cache for chunks
 * of up to n_tokens tokens: 0 for a bf16 cache; for a binary16 cache, the
 * chunk's K and V as stored (2 * n_tokens * n_kv_heads * head_dim * 2
 * bytes); for an fp8 cache, a bf16 image of one sequence's units of the
 * largest layer (K tiles and V rows, the layout of a bf16 cache) plus the
 * chunk's K and V. */
int hwkv_prefill_attn_workspace_bytes(const hwkv_cache *cache, int64_t n_tokens,
                                      size_t *bytes);

/* hwkv_prefill_attn for every cache format.  With an fp8 or binary16 cache
 * the keys and values enter with their stored values -- the cached ones as
 * stored, the chunk's own as the cache will store them -- because a format
 * that changes numerical execution is used by every consumer of the cache
 * (Method, Eq. nominal-storage and the paragraph after it).
 *   fp8: q.k is taken over the decoded codes and multiplied by the K scale,
 *        the output by the V scale.  Every E4M3 value is a bf16 value, so
 *        the codes are staged into ws as bf16 (exactly) and the bf16 MFMA
 *        kernel runs on them.
 *   binary16: the cached rows are read in place and the chunk's rows are
 *        staged into ws as binary16; binary16 MFMA products.  q enters as
 *        binary16 after scaling by a power of two per group of 32
 *        consecutive (token, q head) columns, exact for every component
 *        within a factor 2^31 of the group's largest |q|; the softmax
 *        weights enter the value product rounded to binary16 (with a 2^7
 *        bias that keeps them out of its subnormal range).
 *   ws, ws_bytes  device workspace of >= hwkv_prefill_attn_workspace_bytes
 *                 for n_tokens (may be NULL for a bf16 cache)
 * Other arguments, results and errors as hwkv_prefill_attn; EINVAL for a
 * short or missing workspace. */
int hwkv_prefill_attn_ws(hwkv_cache *cache, int32_t layer, int32_t seq,
                         int64_t pos0, int64_t n_tokens, const void *q,
                         const void *k, const void *v, float scale, void *out,
                         void *ws, size_t ws_bytes, void *stream);

/* Append one token to every sequence of `layer`: token n_b of sequence b
 * goes to slot(n_b) of each unit (once n_b >= S + w this overwrites token
 * n_b - w, the one leaving the window), then n_b += 1.  The window is J_t(w)
 * of Method, Eq. conditional-attention (the last w positions up to the
 * query's own), with the S sinks kept in front; a token is evicted when it
 * leaves that set, as the sink-plus-recent cache of the Appendix evicts once
 * it holds S + w tokens.  ENOMEM if a paged cache's pool has too few pages
 * for the tokens.
 *   k_new, v_new   device bf16 [batch][n_kv_heads][head_dim], stored in
 *                  the cache's format.
 * ECAPACITY if a full unit of the layer already holds max_ctx tokens. */
int hwkv_append(hwkv_cache *cache, int32_t layer, const void *k_new,
                const void *v_new, void *stream);

/* Workspace bytes hwkv_decode_attn / hwkv_append_decode_attn need for any
 * layer at any length up to max_ctx (split partials). */
int hwkv_decode_workspace_bytes(const hwkv_cache *cache, size_t *bytes);

/* Decode attention of `layer` over the current residency (Eqs.
 * conditional-attention-weight and conditional-attention with the exact
 * scaled dot product z = scale * q.k): for sequence b and query head qh,
 * out = sum_s softmax_s(z) v_s over the tokens resident in KV head
 * qh / G, i.e. R(n_b) -- call after hwkv_append for the query's own token.
 *   q     device bf16 [batch][n_q_heads][head_dim]
 *   out   device fp32 [batch][n_q_heads][head_dim] (pre-gate, heads
 *         concatenated)
 *   ws    device workspace of ws_bytes >= hwkv_decode_workspace_bytes
 * EINVAL if a sequence is empty or the workspace is short.  Does not change
 * state.  Fp32 accumulation; the result does not depend on the slot order.
 * Keys and values enter with their stored values: for fp8, q.k is taken over
 * the decoded codes and multiplied by the K scale, and the output by the V
 * scale, and the softmax weights enter the value product as two bf16 terms
 * (round(p) and round(p - round(p))), which carry each weight to 2^-18 of
 * itself; for binary16, q enters q.k as binary16 after a power-of-two scaling
 * per query head, exact for every component within a factor 2^31 of the
 * head's largest |q| (the products are exact, the sums fp32). */
int hwkv_decode_attn(hwkv_cache *cache, int32_t layer, const void *q,
                     float scale, void *out, void *ws, size_t ws_bytes,
                     void *stream);

/* hwkv_append followed by hwkv_decode_attn, in one pass over the cache: the
 * new token is attended from k_new/v_new and written to its slot by the same
 * kernel.  Same arguments, errors and result as the two calls in sequence. */
int hwkv_append_decode_attn(hwkv_cache *cache, int32_t layer,
                            const void *k_new, const void *v_new,
                            const void *q, float scale, void *out, void *ws,
                            size_t ws_bytes, void *stream);

/* hwkv_append_decode_attn for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument; the split partials go to a static
 * device array of the library, 16 MiB per device, held until the process
 * ends.  The call itself allocates nothing (no hipMalloc, hipFree or
 * allocating library routine); its first call on a device looks up the
 * array's device address.  Same arguments, kernels, errors and result as
 * hwkv_append_decode_attn, plus EINVAL, with nothing changed, if the call
 * would need more than the 16 MiB of partials (hwkv_decode_workspace_bytes
 * bounds the need of any call on a cache).  Every call on a device shares
 * that device's array: calls that overlap on one device (concurrent
 * streams, several host threads) race on it and must not be issued. */
int hwkv_append_decode_attn_noalloc(hwkv_cache *cache, int32_t layer,
                                    const void *k_new, const void *v_new,
                                    const void *q, float scale, void *out,
                                    void *stream);

/* ------------------------------------------------------------------------ */
/* Calibration (Method, "Sequential Prefix-Conditioned Calibration";         */
/* Appendix, "Calibration Score and Fixed-Prefix Selection" and             */
/* "Finite-grid budget selection")                                           */
/* ------------------------------------------------------------------------ */

/* Device workspace bytes hwkv_calib_replay needs for n_rows sampled rows of
 * an n_hist-token trace: the row positions and ceil(n_hist / 4096) + 3 sets
 * of n_rows x n_q_heads x (head_dim + 4) fp32 partials -- one per split of
 * the keys (at most 4,096 keys each), one for the sinks, and two for the
 * candidates' edge (m, l) pairs.  Independent of the number of windows. */
int hwkv_calib_workspace_bytes(int32_t n_q_heads, int32_t head_dim,
                               int32_t n_sinks, int64_t n_hist, int64_t n_rows,
                               size_t *bytes);

/* Candidate replay of one traced layer.  For every sampled query row r (at
 * position rows[r]) and query head qh of KV head qh / G, the output over
 * R(t + 1) restricted to [0, t] (t = rows[r], n_sinks sinks plus the last w
 * positions) for every finite codebook window w (Eq. conditional-attention,
 * z = scale * q.k), and for the full history; then the stabilised cosine of
 * each candidate against the full output (Eq. stabilized-cosine) and, per
 * KV head, its mean over the rows and the head's G query heads (Eq.
 * conditional-similarity).
 *   windows   host int64 [n_windows], finite (> 0), strictly increasing:
 *             the codebook in order; the full candidate is implicit
 *   k, v      device bf16 [n_hist][n_kv_heads][head_dim]: the layer's traced
 *             full-history keys (post-RoPE) and values
 *   rows      host int64 [n_rows], strictly increasing, in [0, n_hist);
 *             read before the call returns (the library copies them into
 *             pinned memory of its own and from there, on `stream`, into ws)
 *   q         device bf16 [n_rows][n_q_heads][head_dim]: traced queries
 *   outs      device fp32 [n_windows + 1][n_rows][n_q_heads][head_dim]:
 *             the candidate outputs in codebook order, the full one last
 *   scores    device fp32 [n_windows][n_rows][n_q_heads]
 *   means     device fp32 [n_windows][n_kv_heads]
 *   ref_full  device fp32 [n_rows][n_q_heads][head_dim] or NULL: the traced
 *             full-history output; if given, check[r][qh] is the stabilised
 *             cosine of the replayed full output against it (the full-window
 *             check; the paper's runs abort below 0.99)
 *   check     device fp32 [n_rows][n_q_heads], required iff ref_full
 *   ws        device workspace of ws_bytes >= hwkv_calib_workspace_bytes
 * One pass over the trace serves every candidate: the windows are nested
 * suffixes of each row's history (plus the common sinks), so each row's keys
 * are visited once, from the row's position down, and each window's share
 * is taken where the walk crosses the window's edge; a merge then assembles
 * the candidates.  Same arithmetic as hwkv_prefill_attn (bf16 MFMA, fp32
 * accumulation; the weights enter the value product rounded to bf16 under a
 * shift shared by all candidates); scores and means in fp32.  outs is also
 * used as scratch before the merge writes it.  Waits for the stream once
 * (the row positions are uploaded from host memory).  EINVAL on bad shapes,
 * rows or windows, or if (n_windows + 1) * n_rows * n_q_heads >= 2^31. */
int hwkv_calib_replay(int32_t n_kv_heads, int32_t n_q_heads, int32_t head_dim,
                      int32_t n_sinks, int32_t n_windows,
                      const int64_t *windows, int64_t n_hist, const void *k,
                      const void *v, int64_t n_rows, const int64_t *rows,
                      const void *q, float scale, void *outs, void *scores,
                      void *means, const void *ref_full, void *check, void *ws,
                      size_t ws_bytes, void *stream);

/* hwkv_calib_workspace_bytes for hwkv_calib_replay_format: the same, plus
 * for an fp8 format the trace's K and V staged as bf16 code values
 * (2 * n_hist * n_kv_heads * head_dim * 2 bytes). */
int hwkv_calib_workspace_bytes_format(int32_t n_kv_heads, int32_t n_q_heads,
                                      int32_t head_dim, int32_t n_sinks,
                                      int64_t n_hist, int64_t n_rows,
                                      int32_t kv_format, size_t *bytes);

/* hwkv_calib_replay under cache format kv_format.  When the format changes
 * numerical execution, the full-cache reference, the compressed policy and
 * the calibration scores all use it (Method, the paragraph after Eq.
 * nominal-storage): every candidate, the full one included, attends over the
 * trace's keys and values as a cache of that format stores them, code(x / s)
 * with the per-KV-head fp32 scales k_scale, v_scale [n_kv_heads] (NULL =
 * 1.0; fp8 only).  bf16 is hwkv_calib_replay; EINVAL for binary16.  ws of
 * at least hwkv_calib_workspace_bytes_format bytes. */
int hwkv_calib_replay_format(int32_t n_kv_heads, int32_t n_q_heads,
                             int32_t head_dim, int32_t n_sinks,
                             int32_t n_windows, const int64_t *windows,
                             int64_t n_hist, const void *k, const void *v,
                             int64_t n_rows, const int64_t *rows, const void *q,
                             float scale, void *outs, void *scores, void *means,
                             const void *ref_full, void *check,
                             int32_t kv_format, const float *k_scale,
                             const float *v_scale, void *ws, size_t ws_bytes,
                             void *stream);

/* Eq. threshold-selection for one layer (host only): for each KV head h, the
 * codebook candidate of lowest cost min(n_sinks + w, ctx) whose mean score
 * means[k][h] is at least tau; equal costs go to the earlier codebook entry;
 * the full candidate (score one, cost ctx) is last in the codebook and
 * always feasible.  choice[h] receives the window index, or n_windows for
 * full; *floor (if non-NULL) the lowest selected mean (1 for full), whose
 * minimum over layers is a run's floor. */
int hwkv_calib_select(int32_t n_kv_heads, int32_t n_windows,
                      const int64_t *windows, int32_t n_sinks, int64_t ctx,
                      const double *means, double tau, int32_t *choice,
                      double *floor);

/* Eq. budget-selector over a recorded grid of n_records runs (host only):
 * among runs g with rates[g] <= budget, the largest floors[g], then the
 * smallest rate, then the smallest g.  *chosen = g, or -1 if no run meets
 * the budget. */
int hwkv_budget_select(int32_t n_records, const double *rates,
                       const double *floors, double budget, int32_t *chosen);

/* Calibration artifact (Appendix, experimental protocol: each run stores its
 * artifact identifier, seed and final policy matrix; Appendix, finite-grid
 * budget selection: run g is recorded as (g, tau_g, policy, rate, floor)).
 * Text (JSON) of one object with the keys "format" ("hwkv-policy/1"),
 * "artifact", "seed", "grid_index", "tau", "rate", "floor", "n_layers",
 * "n_kv_heads", "n_q_heads", "head_dim", "n_sinks", "level_window" and
 * "level_of_unit" ([n_layers][n_kv_heads]); doubles carry 17 significant
 * digits, so they read back bit for bit.  Host only.
 *
 * Serialise: artifact_id is printable ASCII without '"' or '\\' (EINVAL
 * otherwise).  *len receives the text length (without the terminating NUL);
 * buf == NULL queries it; a buf of cap < *len + 1 bytes gets ENOMEM. */
int hwkv_policy_serialize(const hwkv_policy *policy, const char *artifact_id,
                          uint64_t seed, int32_t grid_index, double tau,
                          double rate, double floor, char *buf, size_t cap,
                          size_t *len);

/* Parse an artifact written by hwkv_policy_serialize: a new policy in *out
 * (validated as by hwkv_policy_set) and the recorded fields (each output
 * pointer may be NULL; artifact_id receives at most id_cap - 1 characters
 * and a NUL).  EINVAL on any other text: unknown, missing or repeated keys,
 * malformed values, strings with escapes or characters outside printable
 * ASCII, trailing characters. */
int hwkv_policy_deserialize(const char *buf, size_t len, hwkv_policy **out,
                            char *artifact_id, size_t id_cap, uint64_t *seed,
                            int32_t *grid_index, double *tau, double *rate,
                            double *floor);

/* Kernel timing, for profiling.  While enabled (enable != 0) on a cache,
 * every hwkv_decode_attn / hwkv_append_decode_attn call launches its split
 * and merge kernels with start and stop HIP events (hipExtLaunchKernel), per
 * launch group, so that each event pair spans the kernel's own execution and
 * not its dispatch.  Timed launches take profiling work on the stream; leave
 * timing disabled when measuring end-to-end time.  Disabling keeps what was
 * recorded. */
int hwkv_decode_timing(hwkv_cache *cache, int32_t enable);

/* Waits for the recorded calls to complete and returns the summed durations
 * of their split kernels and merge kernels in milliseconds and the number
 * of kernel launch groups recorded, then clears the record. */
int hwkv_decode_timing_read(hwkv_cache *cache, double *split_ms,
                            double *merge_ms, int64_t *launches);

/* Test hook: synchronously copy unit (layer, kv_head) of sequence `seq` to
 * the host after all device work completes.  host_k, host_v receive
 * [capacity][head_dim] stored elements in slot order (bf16 or binary16 bit
 * patterns, 2 bytes each, or E4M3 codes, 1 byte each); *n_valid =
 * min(n, capacity), the number of occupied slots.  Slots >= n_valid hold
 * unspecified values. */
int hwkv_cache_read_unit(const hwkv_cache *cache, int32_t layer,
                         int32_t kv_head, int32_t seq, void *host_k,
                         void *host_v, int64_t *n_valid);

#ifdef __cplusplus
}
#endif

#endif /* HWKV_H */
