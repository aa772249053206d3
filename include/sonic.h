/*
 * sonic.h - C ABI of the SONIC segment-structured attention path on MI355X (gfx950).
 *
 * SONIC (Segmented Optimized Nexus for Information Compression) inserts Nexus
 * tokens after every history segment of a multi-turn conversation, restricts
 * attention with a hierarchical visibility mask, then keeps only the system
 * prompt, the Nexus tokens and the current query in the KV cache.  This
 * library runs the three steps of that path on one GPU:
 *
 *   sonic_segment_attn_prefill  - attention over the augmented sequence of
 *                                 Eq.(1) under the mask of Sec. 3.2, Eqs.(3)-(5);
 *   sonic_kv_compact            - the KV retention rule (Sec. 3, Fig. 2 caption;
 *                                 Sec. 3.2 after Eq.(4); App. C);
 *   sonic_compressed_decode     - one generation step over the retained context
 *                                 {I_sys, N, Q_n} (App. C, Eq.(15));
 *   sonic_nexus_extend          - when a turn ends, the Nexus tokens of its
 *                                 segments (utterance, response) over the
 *                                 compact cache, each segment's rows replaced by
 *                                 its Nexus KV (Sec. 3.2; the Nexus KV is kept
 *                                 for the rest of the session).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers marked "device" are HIP device pointers; "host" pointers are CPU
 *   memory.  The caller owns every buffer.  The three GPU calls never allocate,
 *   free or synchronise: all work is enqueued on `stream` (a hipStream_t; NULL is
 *   the default stream).
 * - Tensors are token-major and packed over the batch ("varlen"): request b owns
 *   rows cu_seqlens[b] .. cu_seqlens[b+1]-1.  Q is bf16 [T][Hq][d]; K and V are
 *   bf16 [T][Hkv][d]; outputs are fp32 [T][Hq][d].  bf16 values are passed as
 *   raw 16-bit patterns.  Rows are contiguous (no strides).
 * - Grouped-query attention: q-head h reads kv-head h / (Hq / Hkv).
 * - Roles (one byte per token): SONIC_ROLE_*.  turn_id is the history segment
 *   index: constant within a segment (its body and its Nexus tokens), strictly
 *   increasing from one history segment to the next, ignored for system and
 *   current tokens.  A request must read
 *       SYSTEM* ( HISTORY_TEXT+ NEXUS* )* CURRENT*
 *   (Eq.(1)); anything else is a layout error.  A segment may have zero Nexus
 *   tokens; it then ends at its last body token.
 * - Synchronous errors (bad arguments, unsupported shapes, small workspace) are
 *   returned before anything is enqueued; outputs are untouched.
 * - Asynchronous errors (layout grammar, cache capacity, a size argument the
 *   device data contradicts) are found by the kernels and written to the device
 *   word *dev_status (first error wins).  The caller zeroes *dev_status before
 *   first use.  While it is non-zero every later kernel of this library that
 *   receives it returns without writing its outputs, so an error is sticky until
 *   the caller clears it.  The one exception is a pending SONIC_ERR_CAPACITY in
 *   sonic_compressed_decode, where capacity is a per-request matter (see there).
 * - softmax_scale: 0 selects the standard scale 1/sqrt(head_dim); any other value
 *   must be finite and positive.
 * - Setting the environment variable SONIC_DEBUG_SYNC=1 makes each GPU call
 *   synchronise its stream and return the device status (debugging only).
 * - Thread safety: calls are independent; the library keeps no mutable global
 *   state apart from a per-device cache of launch parameters.
 */
#ifndef SONIC_H
#define SONIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    SONIC_OK = 0,
    SONIC_ERR_INVALID_ARG = 1,   /* null pointer, negative or inconsistent size      */
    SONIC_ERR_BAD_LAYOUT = 2,    /* role / turn_id sequence breaks the Eq.(1) order  */
    SONIC_ERR_CAPACITY = 3,      /* a request needs more cache rows than it owns     */
    SONIC_ERR_WORKSPACE = 4,     /* workspace smaller than the *_workspace_bytes()   */
    SONIC_ERR_UNSUPPORTED = 5,   /* head_dim not in {64,128}, Hq/Hkv > 8, ...        */
    SONIC_ERR_HIP = 6            /* a HIP runtime call failed                        */
};

enum {
    SONIC_ROLE_SYSTEM = 0,       /* I_sys                                            */
    SONIC_ROLE_HISTORY_TEXT = 1, /* body B_i of a history segment m_i                */
    SONIC_ROLE_NEXUS = 2,        /* Nexus token of N_i                               */
    SONIC_ROLE_CURRENT = 3       /* Q_curr, and every generated token                */
};

/*
 * Scope of Nexus <-> Nexus visibility in the prefill mask.
 *   SONIC_NEXUS_ALL        Eq.(5) as written: every Nexus token sees every Nexus
 *                          token of the request, within and across segments.
 *   SONIC_NEXUS_UP_TO_OWN  a Nexus token sees the Nexus tokens of its own segment
 *                          and of the earlier ones only.  This is what a session
 *                          computes when each segment's Nexus tokens are made as
 *                          its turn ends, over the Nexus KV kept from the earlier
 *                          turns (sonic_nexus_extend); a full prefill with this
 *                          scope reproduces those rows.
 * Every other rule of the mask is the same under both.
 */
enum {
    SONIC_NEXUS_ALL = 0,
    SONIC_NEXUS_UP_TO_OWN = 1
};

/* Version of this ABI (bumped on any signature or layout change or addition). */
int32_t sonic_abi_version(void);

/* Static text for a status code. */
const char *sonic_status_string(int32_t status);

/* ------------------------------------------------------------------------ */
/* Host-side helpers (pure CPU, no GPU needed)                               */
/* ------------------------------------------------------------------------ */

/*
 * Check the layout grammar of a packed batch (Eq.(1), Sec. 3.1) on the CPU.
 * cu_seqlens: host [batch+1]; role, turn_id: host [cu_seqlens[batch]].
 * Returns SONIC_OK or SONIC_ERR_BAD_LAYOUT (then *bad_request, if non-NULL,
 * receives the first failing request) or SONIC_ERR_INVALID_ARG.
 */
int32_t sonic_validate_layout_host(int32_t batch, const int32_t *cu_seqlens, const uint8_t *role,
                                   const int32_t *turn_id, int32_t *bad_request);

/*
 * Per-request work figures of a well-formed batch, on the CPU:
 *   visible_pairs[b] - number of (query, key) pairs the mask of Sec. 3.2 leaves
 *                      visible under nexus_scope (SONIC_NEXUS_*); prefill does
 *                      4*d flops per pair and q-head;
 *   kept_rows[b]     - rows retained by compaction (system + Nexus + current).
 * Either output may be NULL.  Returns SONIC_ERR_BAD_LAYOUT on a grammar error,
 * SONIC_ERR_INVALID_ARG for an unknown scope.
 */
int32_t sonic_layout_stats_host(int32_t batch, const int32_t *cu_seqlens, const uint8_t *role,
                                const int32_t *turn_id, int32_t nexus_scope, int64_t *visible_pairs,
                                int32_t *kept_rows);

/* ------------------------------------------------------------------------ */
/* Step 1: masked prefill attention                                          */
/* ------------------------------------------------------------------------ */

/*
 * Bytes of device workspace sonic_segment_attn_prefill needs for this batch
 * (0 for negative sizes or non-positive heads / head_dim).  It holds the
 * per-block plan, a copy of each request's system and Nexus K/V rows, and the
 * buffers of the attention statistics, so it grows as
 * total_tokens * (num_kv_heads * head_dim * 4 + (num_q_heads + num_kv_heads) * 4)
 * bytes.
 */
size_t sonic_prefill_workspace_bytes(int32_t batch, int32_t total_tokens, int32_t num_q_heads,
                                     int32_t num_kv_heads, int32_t head_dim);

/*
 * out[p][h] = sum_q softmax_q(scale * <q[p][h], k[q][g(h)]> + M[p][q]) * v[q][g(h)]
 * for every token p of every request, where M is the hierarchical visibility
 * mask of Sec. 3.2: causal (Eq.(3), applied globally), history bodies removed
 * for every position after their segment's last Nexus token (Eq.(4)), and
 * Nexus tokens mutually visible (Eq.(5)): all of them under SONIC_NEXUS_ALL,
 * those of the own and earlier segments under SONIC_NEXUS_UP_TO_OWN.
 * Fully masked key blocks are never visited: the kernels enumerate the visible
 * keys of each block of query rows from the segment structure.
 *
 *   batch, total_tokens   B and T = cu_seqlens[B] (host values)
 *   num_q_heads/kv_heads  Hq, Hkv; Hq % Hkv == 0 and Hq / Hkv <= 8
 *   head_dim              d in {64, 128}
 *   cu_seqlens            device int32 [B+1], non-decreasing, cu[0] = 0
 *   role, turn_id         device uint8 [T], int32 [T]
 *   q                     device bf16 [T][Hq][d];  k, v: device bf16 [T][Hkv][d]
 *   softmax_scale         0 for 1/sqrt(d), else finite and > 0
 *   nexus_scope           SONIC_NEXUS_ALL or SONIC_NEXUS_UP_TO_OWN
 *   out                   device fp32 [T][Hq][d] (fully written on success)
 *   nexus_mass            NULL, or device fp32 [T][Hq]: per row p and q-head h the
 *                         attention mass on the request's Nexus keys,
 *                         sum over Nexus keys x of softmax_x(...)[p][x] (the
 *                         quantity the Nexus attention regulariser of Sec. 4
 *                         averages over the current query)
 *   key_weight            NULL, or device fp32 [T]: per key x the attention it
 *                         receives from the CURRENT rows of its request, summed
 *                         over those rows and averaged over the q-heads (the
 *                         importance score of the attention-guided distillation
 *                         of Sec. 4); 0 for history-body keys, which no current
 *                         row sees.  Deterministic (no atomic sums).
 *                         Either statistic costs a few percent of the prefill.
 *   workspace             device, >= sonic_prefill_workspace_bytes(B, T, Hq, Hkv, d) bytes,
 *                         256-byte aligned; contents need no initialisation
 *   dev_status            device int32 (see conventions); SONIC_ERR_BAD_LAYOUT
 *                         is reported here and then no output is written
 * Returns SONIC_ERR_UNSUPPORTED when T * Hkv * d * 2 bytes (one of k, v) reach
 * 4 GiB or T * Hq * d reaches 2^40.
 */
int32_t sonic_segment_attn_prefill(int32_t batch, int32_t total_tokens, int32_t num_q_heads,
                                   int32_t num_kv_heads, int32_t head_dim, const int32_t *cu_seqlens,
                                   const uint8_t *role, const int32_t *turn_id, const void *q, const void *k,
                                   const void *v, float softmax_scale, int32_t nexus_scope, float *out,
                                   float *nexus_mass, float *key_weight, void *workspace, size_t workspace_bytes,
                                   int32_t *dev_status, void *stream);

/* ------------------------------------------------------------------------ */
/* Role-routed linear layer (the projections around the attention)          */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace sonic_role_projection needs (0 for T < 0). */
size_t sonic_role_projection_workspace_bytes(int32_t total_tokens);

/*
 * y[t] = W_N x[t] for every Nexus row t, y[t] = W x[t] for every other row
 * (system, history text, current, generated): Nexus tokens have their own
 * projection matrices and MLP branches (Sec. 3.1), so every linear layer of
 * the block is this routed product with that layer's two weight sets.
 *
 *   total_tokens    T (host value), any T >= 0
 *   in_features     K, a positive multiple of 64
 *   out_features    N >= 1
 *   role            device uint8 [T] (SONIC_ROLE_*); rows are routed by it alone
 *   x               device bf16 [T][K]
 *   w_text, w_nexus device bf16 [N][K] each (output-by-input, as a linear layer stores it)
 *   y               device fp32 [T][N], every row written
 *   workspace       device, >= sonic_role_projection_workspace_bytes(T), 256-byte aligned
 *   dev_status      device int32; while it is non-zero nothing is written
 * Products are accumulated in fp32 from exact bf16 products.
 * Returns SONIC_ERR_UNSUPPORTED when K is not a multiple of 64, or when x or one
 * weight set spans more than 4 GiB (T * K * 2 or N * K * 2 bytes).
 */
int32_t sonic_role_projection(int32_t total_tokens, int32_t in_features, int32_t out_features,
                              const uint8_t *role, const void *x, const void *w_text, const void *w_nexus,
                              float *y, void *workspace, size_t workspace_bytes, int32_t *dev_status,
                              void *stream);

/* ------------------------------------------------------------------------ */
/* Reconstruction targets of the Nexus tokens (training side)                */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace sonic_nexus_recon_targets needs (0 for negative sizes). */
size_t sonic_nexus_recon_workspace_bytes(int32_t batch, int32_t total_tokens);

/*
 * Per Nexus token, the reconstruction target of the information bottleneck
 * (Sec. 4): the body of its history segment is cut into one sub-interval per
 * Nexus token of the segment, interval j of a b-token body for K Nexus tokens
 * being [floor(j b / K), max(floor((j + 1) b / K), floor(j b / K) + 1)) (near-
 * equal pieces; single tokens when b < K), and
 *     target_j = sum over x of alpha(x) h(x),  alpha = softmax over x of cos(h(N_j), h(x)).
 * A zero vector has cosine 0 with anything.
 *
 *   batch, total_tokens   B, T (host values)
 *   hidden                hidden size Dm: a positive multiple of 8, at most 16384
 *   cu_seqlens, role, turn_id   device, the layout as for the prefill
 *   h                     device bf16 [T][Dm]: the hidden states
 *   max_rows              rows of the three outputs (>= the batch's Nexus count)
 *   target                device fp32 [n][Dm]: one row per Nexus token of the batch,
 *                         in packed position order
 *   cos_target            device fp32 [n]: cos(h(N_j), target_j)
 *   entropy_ratio         device fp32 [n]: H(alpha) / log |interval| (1 for one token)
 *   workspace             device, >= sonic_nexus_recon_workspace_bytes(B, T), 256-byte aligned
 *   dev_status            device int32: SONIC_ERR_BAD_LAYOUT for a grammar error,
 *                         SONIC_ERR_CAPACITY when the Nexus count exceeds max_rows;
 *                         then nothing is written
 * Reproducible: the reductions run in a fixed order.
 */
int32_t sonic_nexus_recon_targets(int32_t batch, int32_t total_tokens, int32_t hidden,
                                  const int32_t *cu_seqlens, const uint8_t *role, const int32_t *turn_id,
                                  const void *h, int32_t max_rows, float *target, float *cos_target,
                                  float *entropy_ratio, void *workspace, size_t workspace_bytes,
                                  int32_t *dev_status, void *stream);

/* ------------------------------------------------------------------------ */
/* Step 2: KV compaction                                                     */
/* ------------------------------------------------------------------------ */

/*
 * Keep the K/V rows of every token whose role is not HISTORY_TEXT, in order
 * (system prompt, Nexus tokens, current query; Sec. 3, Fig. 2 caption).
 * Request b's j-th kept token goes to cache row cache_row_off[b] + j, bit for
 * bit; keep_idx at that row receives its request-local source position; and
 * cache_len[b] receives the kept count.  Rows from the kept count up to the
 * request's capacity are not written.
 *
 *   batch, total_tokens, max_seqlen  host values; max_seqlen >= every request length
 *                                    (the grid is sized from it: a longer request
 *                                    raises SONIC_ERR_INVALID_ARG on the device and
 *                                    none of its rows is written)
 *   num_kv_heads, head_dim           Hkv, d (d in {64, 128})
 *   cu_seqlens, role                 device, as for the prefill; role 16-byte
 *                                    aligned (it is read in 16-byte words, never
 *                                    past its total_tokens bytes)
 *   k, v                             device bf16 [T][Hkv][d]
 *   k_cache, v_cache                 device bf16 [rows][Hkv][d]
 *   cache_row_off                    device int64 [B]: first cache row of request b
 *   cache_row_cap                    device int32 [B]: rows request b owns
 *   cache_len                        device int32 [B], written
 *   keep_idx                         device int32 [rows], written at kept rows
 *   dev_status                       device int32; SONIC_ERR_CAPACITY when a
 *                                    request keeps more rows than its capacity
 *                                    (no row beyond the capacity is written)
 */
int32_t sonic_kv_compact(int32_t batch, int32_t total_tokens, int32_t max_seqlen, int32_t num_kv_heads,
                         int32_t head_dim, const int32_t *cu_seqlens, const uint8_t *role, const void *k,
                         const void *v, void *k_cache, void *v_cache, const int64_t *cache_row_off,
                         const int32_t *cache_row_cap, int32_t *cache_len, int32_t *keep_idx,
                         int32_t *dev_status, void *stream);

/* ------------------------------------------------------------------------ */
/* Step 3: decode over the compacted cache                                   */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace sonic_compressed_decode needs (any Hkv dividing Hq). */
size_t sonic_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t head_dim, int32_t max_ctx);

/*
 * One generation step for every request b (App. C, Eq.(15)): the new token's
 * k_new[b], v_new[b] are appended at cache row cache_row_off[b] + cache_len[b],
 * then
 *     out[b][h] = softmax(scale * q[b][h] . Kc^T) Vc
 * over the request's rows 0 .. cache_len[b] (the appended row included): a
 * generated token belongs to the current turn, so it sees every retained row.
 * cache_len[b] is incremented on the device, so a decode loop needs no host
 * round trip.  One kernel: the context of each (request, kv-head) is split over
 * up to min(16, 256 / (B * Hkv)) workgroups (three for 256 or more pairs with
 * contexts of 2048 rows and more), and the split that finishes last merges the
 * partials by log-sum-exp.
 *
 * With row_role == NULL the cache is a compact one and every row is visible.
 * With row_role != NULL (device uint8 [rows], indexed like cache rows) the
 * cache is a full, uncompacted one: rows whose role is HISTORY_TEXT are masked
 * (Eq.(4)); the caller marks rows appended by earlier steps as CURRENT.
 *
 *   max_ctx        host bound: cache_len[b] + 1 <= max_ctx for every b
 *   q              device bf16 [B][Hq][d];  k_new, v_new: device bf16 [B][Hkv][d]
 *   out            device fp32 [B][Hq][d]
 *   workspace      device, 256-byte aligned, >= sonic_decode_workspace_bytes(B, Hq, d,
 *                  max_ctx); zero-filled before its first use (it holds completion
 *                  counters that every call leaves at zero again)
 *   dev_status     SONIC_ERR_CAPACITY when cache_len[b] + 1 exceeds the capacity
 *                  or max_ctx: request b is then left unchanged (no append, no
 *                  output, same length) while the other requests proceed.
 *                  Capacity is per request, so a pending SONIC_ERR_CAPACITY does
 *                  not stop later decode calls either (each full request keeps
 *                  failing on its own).  Any other pending error (a layout or
 *                  argument error of an earlier call) stops the call: nothing is
 *                  appended, written or advanced for any request.
 * Calls that share a workspace must not run concurrently.
 */
int32_t sonic_compressed_decode(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                int32_t max_ctx, void *k_cache, void *v_cache, const int64_t *cache_row_off,
                                const int32_t *cache_row_cap, int32_t *cache_len, const uint8_t *row_role,
                                const void *q, const void *k_new, const void *v_new, float softmax_scale,
                                float *out, void *workspace, size_t workspace_bytes, int32_t *dev_status,
                                void *stream);

/*
 * The same decode step as sonic_compressed_decode, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): no workspace argument, and the call allocates nothing.  Its
 * completion counters and split partials live in one fixed device array of 8 MiB per
 * GPU that the library holds until the process ends; the counters sit in its first
 * 64 KiB, at the same place for every call, and every call leaves them at zero (the
 * first call on a GPU also enqueues a small kernel on `stream` that clears them).
 * Arguments, outputs and errors are those of sonic_compressed_decode, plus:
 *   - SONIC_ERR_WORKSPACE (returned, nothing enqueued) when the call needs more than
 *     the array holds: batch > 4096, batch * num_kv_heads > 12288, or more than
 *     8 MiB - 64 KiB of partials (batch * num_q_heads * splits * (head_dim + 2) * 4 B,
 *     splits as sonic_decode_workspace_bytes counts them);
 *   - calls on one GPU share the array, so calls that overlap on it (concurrent
 *     streams, other threads) race; calls ordered on one stream do not.
 */
int32_t sonic_compressed_decode_noalloc(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                        int32_t head_dim, int32_t max_ctx, void *k_cache, void *v_cache,
                                        const int64_t *cache_row_off, const int32_t *cache_row_cap,
                                        int32_t *cache_len, const uint8_t *row_role, const void *q,
                                        const void *k_new, const void *v_new, float softmax_scale, float *out,
                                        int32_t *dev_status, void *stream);

/* ------------------------------------------------------------------------ */
/* Next turn: the ended turn's Nexus tokens over the compact cache            */
/* ------------------------------------------------------------------------ */

/*
 * Bytes of device workspace sonic_nexus_extend needs (0 for negative sizes or
 * non-positive heads / head_dim): the plan, and room to stage up to max_rows rows of
 * K and V per request (the tail rows after a segment body, see body_len).
 */
size_t sonic_nexus_extend_workspace_bytes(int32_t batch, int32_t total_new, int32_t max_rows,
                                          int32_t num_kv_heads, int32_t head_dim);

/*
 * When turn n of request b ends, its rows (query and generated response) are the
 * last rows of the request's compact cache, rows keep_len[b] .. cache_len[b]-1.  Each
 * user utterance and each assistant response is a history segment of its own, with
 * its own Nexus tokens (Eq.(1), Sec. 3.1); one call computes the Nexus tokens of one
 * segment per request, whose body is the first body_len[b] of those rows (all of
 * them when body_len is NULL).  For every new Nexus row p and q-head h
 *     out[p][h] = softmax_q(scale * <q[p][h], k[q][g(h)]>) v[q][g(h)]
 * over q in {the request's cache rows 0 .. keep_len[b] + body_len[b] - 1} u {its new
 * Nexus rows}: by Sec. 3.2 a Nexus row of the segment sees the system prompt and the
 * earlier segments' Nexus tokens (Eq.(3)), its own body (Eq.(4)) and all the Nexus
 * tokens of its segment (Eq.(5)), and not the tail rows after the body, which come
 * later (Eq.(3)).  The result does not depend on whether Nexus tokens see later
 * segments' Nexus tokens, since none exist yet: utterance then response, one call
 * each, give what a full prefill with SONIC_NEXUS_UP_TO_OWN gives for both.  Then
 * the new Nexus K/V are written to cache rows keep_len[b] .., over the body, which no
 * later row may see (Eq.(4)); the tail rows after the body follow them unchanged; and
 * cache_len[b] becomes keep_len[b] + (new Nexus rows of b) + (tail rows after the
 * body).  The next segment's call then takes keep_len[b] + (new Nexus rows of b).
 *
 *   batch, total_new   B and N = nexus_cu[B] (host values); a request may have
 *                      no new Nexus rows (its body is then only dropped)
 *   max_rows           host bound: cache_len[b] <= max_rows for every b
 *   nexus_cu           device int32 [B+1], non-decreasing, nexus_cu[0] = 0:
 *                      request b's new Nexus rows are rows nexus_cu[b] .. of q/k/v
 *   keep_len           device int32 [B]: cache rows kept (system prompt and the
 *                      earlier Nexus tokens), 0 <= keep_len[b] <= cache_len[b]
 *   body_len           NULL, or device int32 [B]: rows of the segment's body,
 *                      0 <= body_len[b] <= cache_len[b] - keep_len[b]
 *   k_cache .. cache_len   the compact cache, as for sonic_compressed_decode
 *   q                  device bf16 [N][Hq][d];  k, v: device bf16 [N][Hkv][d]
 *   softmax_scale      0 for 1/sqrt(d), else finite and > 0
 *   out                device fp32 [N][Hq][d]
 *   workspace          device, 256-byte aligned,
 *                      >= sonic_nexus_extend_workspace_bytes(B, N, max_rows, Hkv, d);
 *                      contents need no initialisation
 *   dev_status         SONIC_ERR_BAD_LAYOUT when nexus_cu or the lengths are
 *                      inconsistent, SONIC_ERR_CAPACITY when the new length would
 *                      exceed the capacity; then (as with any pending status)
 *                      nothing is written
 * Returns SONIC_ERR_UNSUPPORTED when max_rows or N rows of one tensor reach 4 GiB.
 */
int32_t sonic_nexus_extend(int32_t batch, int32_t total_new, int32_t num_q_heads, int32_t num_kv_heads,
                           int32_t head_dim, int32_t max_rows, const int32_t *nexus_cu, const int32_t *keep_len,
                           const int32_t *body_len, void *k_cache, void *v_cache, const int64_t *cache_row_off,
                           const int32_t *cache_row_cap, int32_t *cache_len, const void *q, const void *k,
                           const void *v, float softmax_scale, float *out, void *workspace,
                           size_t workspace_bytes, int32_t *dev_status, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SONIC_H */
