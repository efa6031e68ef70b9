/*
 * grace.h -- C ABI of the wide-beam decode attention library for MI355X (gfx950).
 *
 * One decode step of an encoder-decoder generative retriever under beam search
 * (GRACE, arXiv 2608.00938):
 *
 *   grace_cross_attn      the beams of a request attend to that request's shared
 *                         encoder K/V, beam-as-query layout (Sec. 5.1, App. B);
 *   grace_kv_append       paged beam rearrangement: block-table rows copy their
 *                         parent's ids, the current token takes a fresh block
 *                         (Sec. 3.3, Sec. 5.3);
 *   grace_self_attn_step  each beam attends over its short paged Semantic-ID
 *                         prefix, positions 0..step (Sec. 5.2, Sec. 5.3);
 *   grace_self_attn_step_fused
 *                         the previous two in one pass: table update, append
 *                         and self-attention (Sec. 5.2 kernel fusion, Sec. 5.3);
 *                         _dyn: the same with per-step beam widths (Sec. 3.3);
 *   grace_beam_scores     beam score update: prefix score + token log-prob,
 *                         filtered tokens removed (Sec. 3.1);
 *   grace_beam_topk       per-request top-k that yields the next step's beams,
 *                         i.e. the parents the rearrangement consumes (Sec. 3.1,
 *                         Sec. 3.3);
 *   grace_gtm_mask        decode-time constraint filter: constrained decoding on
 *                         the SID trie and target matching (Sec. 4, Sec. 5.4, App. A);
 *   grace_trie_advance    the trie node each selected beam moves to (Sec. 4.4);
 *   grace_graph_*         capture of a sequence of these calls (a whole decode
 *                         loop) as one replayable HIP graph (Sec. 5).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  Pointers documented as "device" are HIP device allocations owned by
 *   the caller.  The library allocates nothing, frees nothing and keeps no
 *   pointer after it returns.
 * Layout.  Row-major and contiguous.  Beam rows are request-major: row
 *   r = b*M + m holds beam m of request b (App. B).  A token vector is [H, d]
 *   (head-major), so a [rows, H, d] tensor has element (r, h, i) at
 *   r*H*d + h*d + i.
 * Types.  dtype is GRACE_F32 (float) or GRACE_BF16 (bfloat16) and applies to
 *   every q/k/v/out/pool argument of the call.  Dot products, softmax and
 *   accumulation run in fp32; outputs are rounded to nearest-even.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = null stream).
 *   Work is enqueued on it and not waited for; the library does no host
 *   synchronisation and holds no global state besides the thread-local last
 *   HIP error, so calls from several threads on several streams are safe
 *   (grace_beam_step_noalloc, which keeps a scratch array per GPU, is the
 *   one exception; see there).
 * Errors.  Every argument check runs on the host before any launch; a
 *   non-zero status means nothing was launched and nothing was written.  A
 *   HIP launch failure returns GRACE_ERR_HIP and grace_last_hip_error() gives
 *   the hipError_t code.  Supported: d in {32, 64, 128}; 1 <= T_max <= 8;
 *   0 <= step < T_max; H >= 1; B, M >= 0 (B*M = 0 is a no-op); B*M*H*d and
 *   T_max*B*M below 2^31.
 */
#ifndef GRACE_H
#define GRACE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum grace_dtype { GRACE_F32 = 0, GRACE_BF16 = 1 };

enum grace_status {
  GRACE_OK = 0,
  GRACE_ERR_NULL = 1,         /* a required pointer is NULL                     */
  GRACE_ERR_SHAPE = 2,        /* a size or index argument is out of range       */
  GRACE_ERR_UNSUPPORTED = 3,  /* dtype or head dim the library does not build   */
  GRACE_ERR_ALIAS = 4,        /* an output overlaps an input it must not        */
  GRACE_ERR_HIP = 5           /* a HIP runtime call failed; see grace_last_hip_error */
};

/*
 * Cross-attention of every beam row against its request's encoder K/V, in the
 * beam-as-query layout (Sec. 5.1; correctness of the layout: App. B).  For
 * request b, head h and beam m:
 *   out[b*M+m, h, :] = sum_j softmax_j(scale * <q[b*M+m, h, :], K[off[b]+j, h, :]>)
 *                      * V[off[b]+j, h, :],   j = 0 .. L_b-1,  L_b = off[b+1]-off[b].
 * The M beams of a request are the query rows of one contraction over K/V that
 * the library reads once per beam tile; Q is read in its beam-major layout,
 * with no permuted copy.
 *
 *   q        device, [B*M, H, d], dtype
 *   enc_k    device, [sum_L, H, d], dtype; the requests' encoder keys packed
 *            without padding, request b at rows off[b] .. off[b+1]-1
 *   enc_v    device, [sum_L, H, d], dtype; values, same packing
 *   enc_off  device, int32 [B+1]; enc_off[0] = 0, non-decreasing,
 *            enc_off[B] = sum_L.  Entries are clamped to [0, sum_L] on the
 *            device, so a bad table cannot read out of bounds (its rows are
 *            then unspecified).  A request with L_b = 0 gets zero output rows.
 *   B, M     requests and beams per request
 *   H, d     heads and head dim (d in {32, 64, 128})
 *   sum_L    total encoder tokens (rows of enc_k / enc_v); >= 0
 *   scale    softmax scale, finite and > 0 (1/sqrt(d) for standard attention)
 *   dtype    GRACE_F32 or GRACE_BF16
 *   out      device, [B*M, H, d], dtype; must not overlap q, enc_k or enc_v
 *   stream   hipStream_t
 */
int32_t grace_cross_attn(const void* q, const void* enc_k, const void* enc_v,
                         const int32_t* enc_off, int32_t B, int32_t M, int32_t H, int32_t d,
                         int32_t sum_L, float scale, int32_t dtype, void* out, void* stream);

/*
 * Paged beam rearrangement and append of the current token at decode step
 * `step` (Sec. 3.3, Sec. 5.3).  The KV pool stores one block per generated
 * token of one beam row, across all heads; block id t*R + r (R = B*M) is slab t,
 * row r of a pool laid out [T_max, R, H, d].  For every row i = b*M + m:
 *   table_next[i, j]    = table_prev[b*M + parents[i], j]   for 0 <= j < step
 *   table_next[i, step] = step*R + i                        (its fresh block)
 *   k_pool[step, i, :, :] = k_new[i],  v_pool[step, i, :, :] = v_new[i]
 * Only block ids move for the prefix; no cached K/V bytes are copied.
 * Columns j > step of table_next are not written.
 *
 *   k_pool, v_pool  device, [T_max, B*M, H, d], dtype
 *   table_prev      device, int32 [B*M, T_max]; read for step > 0 (NULL allowed at step 0)
 *   table_next      device, int32 [B*M, T_max]; written; must not overlap table_prev
 *   parents         device, int32 [B*M]; request-local parent beam in [0, M) of each
 *                   new row (NULL allowed at step 0, where parents are ignored).
 *                   An entry outside [0, M) is clamped into range and sets *err_flag.
 *   k_new, v_new    device, [B*M, H, d], dtype; the current token's key and value.
 *                   A pointer equal to its pool's slab `step` is taken as already
 *                   in place and that copy is skipped; any other overlap with the
 *                   written slab is GRACE_ERR_ALIAS.
 *   B, M, H, d      as for grace_cross_attn
 *   T_max           pool slabs and table columns (1 .. 8)
 *   step            decode step, 0 <= step < T_max
 *   dtype           GRACE_F32 or GRACE_BF16
 *   err_flag        device int32 or NULL; set to 1 when a parent was out of range,
 *                   never cleared by the library
 *   stream          hipStream_t
 */
int32_t grace_kv_append(void* k_pool, void* v_pool, const int32_t* table_prev,
                        int32_t* table_next, const int32_t* parents, const void* k_new,
                        const void* v_new, int32_t B, int32_t M, int32_t H, int32_t d,
                        int32_t T_max, int32_t step, int32_t dtype, int32_t* err_flag,
                        void* stream);

/*
 * Self-attention at decode step `step` over each beam's paged prefix
 * (Sec. 5.2, Sec. 5.3).  Row r gathers the step+1 blocks table[r, 0..step] in
 * prefix order; there is no other mask.  For every row r and head h:
 *   out[r, h, :] = sum_j softmax_j(scale * <q[r, h, :], Kblk(table[r, j])[h, :]>)
 *                  * Vblk(table[r, j])[h, :],   j = 0 .. step
 * where Kblk(id) is k_pool viewed as [T_max*B*M, H, d].  Block ids are clamped
 * into [0, T_max*B*M) on the device, so an unwritten table entry cannot read
 * out of bounds (that row's output is then unspecified).
 *
 *   q               device, [B*M, H, d], dtype
 *   k_pool, v_pool  device, [T_max, B*M, H, d], dtype
 *   table           device, int32 [B*M, T_max]; columns 0..step are read
 *   B, M, H, d      as for grace_cross_attn
 *   T_max, step     as for grace_kv_append
 *   scale           softmax scale, finite and > 0
 *   dtype           GRACE_F32 or GRACE_BF16
 *   out             device, [B*M, H, d], dtype; must not overlap q or the pools
 *   stream          hipStream_t
 */
int32_t grace_self_attn_step(const void* q, const void* k_pool, const void* v_pool,
                             const int32_t* table, int32_t B, int32_t M, int32_t H, int32_t d,
                             int32_t T_max, int32_t step, float scale, int32_t dtype, void* out,
                             void* stream);

/*
 * Fused paged append and self-attention at decode step `step` (the paper's
 * fused, paged self-attention: Sec. 5.2, Sec. 5.3).  One pass computes exactly
 * what grace_kv_append followed by grace_self_attn_step on table_next computes:
 *   table_next[i, j]    = table_prev[b*M + parents[i], j]   for 0 <= j < step
 *   table_next[i, step] = step*R + i
 *   k_pool[step, i] = k_new[i],  v_pool[step, i] = v_new[i]
 *   out[i, h, :] = sum_j softmax_j(scale * <q[i, h, :], K_j[h, :]>) * V_j[h, :],
 *     j = 0 .. step, where K_j/V_j for j < step are the blocks table_next[i, j]
 *     and K_step/V_step are k_new[i]/v_new[i] (taken from the inputs, not
 *     re-read from the pool).
 * Each (row, head) reads its ancestors' blocks once and its current token
 * once, so the slab written by the append is never read back in this step.
 *
 *   q               device, [B*M, H, d], dtype
 *   k_new, v_new    device, [B*M, H, d], dtype; as for grace_kv_append (a pointer
 *                   equal to its pool's slab `step` skips that copy)
 *   k_pool, v_pool  device, [T_max, B*M, H, d], dtype; slabs 0..step-1 read,
 *                   slab `step` written
 *   table_prev      device, int32 [B*M, T_max]; read for step > 0 (NULL allowed at step 0)
 *   table_next      device, int32 [B*M, T_max]; columns 0..step written
 *   parents         device, int32 [B*M]; as for grace_kv_append (NULL allowed at step 0)
 *   B, M, H, d      as for grace_cross_attn
 *   T_max, step     as for grace_kv_append
 *   scale           softmax scale, finite and > 0
 *   dtype           GRACE_F32 or GRACE_BF16
 *   out             device, [B*M, H, d], dtype
 *   err_flag        device int32 or NULL; set to 1 when a parent was out of range
 *                   (it is then clamped into [0, M)), never cleared by the library
 *   stream          hipStream_t
 * Every written range (out, table_next, and each slab that is copied) must be
 * disjoint from every other written range and from every range read (q, k_new,
 * v_new, table_prev, parents, pool slabs 0..step-1); otherwise GRACE_ERR_ALIAS.
 */
int32_t grace_self_attn_step_fused(const void* q, const void* k_new, const void* v_new,
                                   void* k_pool, void* v_pool, const int32_t* table_prev,
                                   int32_t* table_next, const int32_t* parents, int32_t B,
                                   int32_t M, int32_t H, int32_t d, int32_t T_max, int32_t step,
                                   float scale, int32_t dtype, void* out, int32_t* err_flag,
                                   void* stream);

/*
 * grace_self_attn_step_fused with dynamic per-step beam widths (Sec. 3.3): the
 * previous step kept M_prev beams per request, this step keeps M_cur, and the
 * pools reserve R_s rows per slab (R_s >= B*M_cur and >= B*M_prev; slab t holds
 * the B*M_t rows of step t).  With new row r = b*M_cur + j:
 *   table_next[r, j'] = table_prev[b*M_prev + parents[r], j']  for 0 <= j' < step
 *   table_next[r, step] = step*R_s + r
 *   k_pool[step, r] = k_new[r],  v_pool[step, r] = v_new[r]
 * and out is the self-attention over table_next[r, 0..step] as in
 * grace_self_attn_step_fused.  Pools are [T_max, R_s, H, d]; block ids index
 * them as [T_max*R_s, H, d] and are clamped into that range on the device.
 *
 *   q, k_new, v_new, out   device, [B*M_cur, H, d], dtype
 *   table_prev             device, int32 [B*M_prev, T_max] (read for step > 0)
 *   table_next             device, int32 [B*M_cur, T_max]
 *   parents                device, int32 [B*M_cur], request-local parents in [0, M_prev);
 *                          out-of-range entries are clamped and set *err_flag
 *   M_prev                 ignored at step 0; else >= 1
 *   other arguments        as for grace_self_attn_step_fused
 * Limits: T_max*R_s and R_s*H*d below 2^31.  Aliasing rules as for
 * grace_self_attn_step_fused (slab `step` means rows step*R_s .. step*R_s+B*M_cur-1).
 */
int32_t grace_self_attn_step_fused_dyn(const void* q, const void* k_new, const void* v_new,
                                       void* k_pool, void* v_pool, const int32_t* table_prev,
                                       int32_t* table_next, const int32_t* parents, int32_t B,
                                       int32_t M_prev, int32_t M_cur, int32_t R_s, int32_t H,
                                       int32_t d, int32_t T_max, int32_t step, float scale,
                                       int32_t dtype, void* out, int32_t* err_flag, void* stream);

/*
 * Beam score update (Sec. 3.1): every candidate (beam row r, token v) scores
 *   cand[r, v] = prev_scores[r] + log_softmax(logits[r, :])[v]      if allowed
 *   cand[r, v] = -inf                                                if filtered
 * The log-softmax is over the whole vocabulary (the filter removes candidates
 * after the model's distribution is formed; no renormalisation over survivors).
 * Arithmetic in fp32.
 *
 *   logits       device, [R, V], dtype (GRACE_F32 or GRACE_BF16)
 *   prev_scores  device, fp32 [R]; accumulated log-probability of each beam's prefix
 *   mask         device, uint32 [R, ceil(V/32)] or NULL (all allowed): bit (v % 32)
 *                of word v / 32 of row r set = token v allowed for beam r (the
 *                constraint filter's output)
 *   R, V         rows and vocabulary size; R*V below 2^31, V >= 1
 *   cand         device, fp32 [R, V], written; must not overlap the inputs
 *   row_max      device, fp32 [R] or NULL; receives max_v cand[r, v]
 *   stream       hipStream_t
 */
int32_t grace_beam_scores(const void* logits, const float* prev_scores, const uint32_t* mask,
                          int32_t R, int32_t V, int32_t dtype, float* cand, float* row_max,
                          void* stream);

/* Largest k grace_beam_topk accepts. */
int32_t grace_beam_topk_max_k(void);

/* Bytes of device workspace grace_beam_topk needs for B, M, V (-1 if out of range). */
int64_t grace_beam_topk_workspace_bytes(int32_t B, int32_t M, int32_t V);

/*
 * Per-request beam top-k (Sec. 3.1; with dynamic widths k = M_{t+1}, Sec. 3.3).
 * Request b owns candidates cand[b*M + m, v], flat index i = m*V + v.  The k
 * best are selected under a total order: score descending, then flat index
 * ascending (-0 equals +0; NaN ranks below -inf), and are written in that
 * order: for j < k,
 *   parents[b*k + j] = i_j / V   (request-local beam in [0, M): the parent of
 *                                 new beam j, as grace_kv_append and the fused
 *                                 entry points consume it with M_cur = k)
 *   tokens[b*k + j]  = i_j % V,  scores[b*k + j] = cand at i_j (bit-exact)
 * k beams are always produced; when fewer than k candidates are finite the
 * rest are filtered candidates (score -inf, dead beams).
 *
 *   cand       device, fp32 [B*M, V]
 *   row_max    device, fp32 [B*M] or NULL: a speed hint (grace_beam_scores'
 *              row maxima); any values give the same result
 *   B, M, V    requests, beams per request, vocabulary; M*V below 2^31 and
 *              B*M*V below 2^40
 *   k          1 <= k <= min(M*V, grace_beam_topk_max_k())
 *   workspace  device, at least grace_beam_topk_workspace_bytes(B, M, V) bytes,
 *              8-byte aligned, caller-owned; contents on entry are ignored and
 *              on return unspecified; calls that share it must not overlap
 *   parents, tokens   device, int32 [B, k];  scores  device, fp32 [B, k]
 *   stream     hipStream_t
 * Outputs and the workspace must not overlap each other or the inputs; a
 * workspace that is too small or misaligned is GRACE_ERR_SHAPE.
 */
int32_t grace_beam_topk(const float* cand, const float* row_max, int32_t B, int32_t M, int32_t V,
                        int32_t k, void* workspace, int64_t workspace_bytes, int32_t* parents,
                        int32_t* tokens, float* scores, void* stream);

/* Bytes of device workspace grace_beam_step needs for B, M, V (-1 if out of range). */
int64_t grace_beam_step_workspace_bytes(int32_t B, int32_t M, int32_t V);

/*
 * Score update and per-request top-k of one beam step in one call (Sec. 3.1;
 * dynamic widths, Sec. 3.3): the same parents, tokens and scores, bit for bit,
 * as grace_beam_scores on these logits, prev_scores and mask (R = B*M rows)
 * followed by grace_beam_topk on the candidates it writes.  The [R, V]
 * candidate array is never written: each candidate the selection reads is
 * recomputed from its logit with the row's log-sum-exp, which a first pass
 * keeps in the workspace.
 *
 *   logits, prev_scores, mask   as for grace_beam_scores, with R = B*M
 *   B, M, V      requests, beams per request, vocabulary; B*M*V below 2^31
 *   k            1 <= k <= min(M*V, grace_beam_topk_max_k())
 *   dtype        GRACE_F32 or GRACE_BF16 (of the logits)
 *   workspace    device, at least grace_beam_step_workspace_bytes(B, M, V)
 *                bytes, 8-byte aligned, caller-owned; contents on entry are
 *                ignored and on return unspecified; calls that share it must
 *                not overlap
 *   parents, tokens, scores     as for grace_beam_topk
 *   stream       hipStream_t
 * Outputs and the workspace must not overlap each other or the inputs; a
 * workspace that is too small or misaligned is GRACE_ERR_SHAPE.
 */
int32_t grace_beam_step(const void* logits, const float* prev_scores, const uint32_t* mask,
                        int32_t B, int32_t M, int32_t V, int32_t k, int32_t dtype,
                        void* workspace, int64_t workspace_bytes, int32_t* parents,
                        int32_t* tokens, float* scores, void* stream);

/* Largest workspace grace_beam_step_noalloc can serve: 80 MiB, enough for
 * 64 requests x 4096 beams x 512 tokens (70.0 MiB). */
#define GRACE_BEAM_STEP_NOALLOC_MAX_BYTES (80ll << 20)

/*
 * grace_beam_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same parents, tokens and scores, bit for bit, with no workspace
 * argument.  The workspace is a scratch array inside the library, one per GPU,
 * of GRACE_BEAM_STEP_NOALLOC_MAX_BYTES; it is set up on the first call on each
 * GPU (with that GPU current) and held until the process ends.  No call
 * allocates or frees device memory.
 *
 *   arguments   as for grace_beam_step, without workspace and workspace_bytes;
 *               `stream` must belong to the current GPU
 * Returns GRACE_ERR_SHAPE when grace_beam_step_workspace_bytes(B, M, V)
 * exceeds GRACE_BEAM_STEP_NOALLOC_MAX_BYTES (nothing is launched), and the
 * statuses of grace_beam_step otherwise.  All calls on one GPU share its
 * scratch array: calls that overlap in time on one GPU (concurrent streams,
 * other host threads) race and give unspecified results; calls ordered on one
 * stream, or separated by synchronisation, do not.  The array's contents
 * between calls are unspecified and never read before being written.
 */
int32_t grace_beam_step_noalloc(const void* logits, const float* prev_scores,
                                const uint32_t* mask, int32_t B, int32_t M, int32_t V, int32_t k,
                                int32_t dtype, int32_t* parents, int32_t* tokens, float* scores,
                                void* stream);

/*
 * The CD + GTM index (Sec. 4.4, App. A): the SID trie in CSR form.  Node 0 is
 * the root; node i's child entries are [node_offsets[i], node_offsets[i+1]).
 * Entry e leads by token tokens[e] to node child_nodes[e]; its eligibility
 * matchers are row bitmask_index[e] of bitmask_table and row bloom_index[e] of
 * bloom_table (deduplicated tables of packed uint64 words).  Within a node's
 * range tokens are distinct and ascending.  The struct lives in host memory;
 * every pointer in it is a device pointer.
 */
typedef struct grace_gtm_index {
  int32_t vocab;             /* |V|, 1..4096; tokens lie in [0, vocab)             */
  int32_t num_nodes;         /* trie nodes (>= 1)                                  */
  int32_t num_entries;       /* child entries (>= 0)                               */
  int32_t bitmask_words;     /* W_bm, 1..8 words per bitmask row                   */
  int32_t bloom_words;       /* W_bl, 1..4 words per Bloom row                     */
  int32_t bitmask_rows;      /* rows of bitmask_table                              */
  int32_t bloom_rows;        /* rows of bloom_table                                */
  int32_t reserved;          /* must be 0                                          */
  const int32_t* node_offsets;   /* int32 [num_nodes + 1]                          */
  const int32_t* child_nodes;    /* int32 [num_entries]                            */
  const int16_t* tokens;         /* int16 [num_entries]                            */
  const int32_t* bitmask_index;  /* int32 [num_entries]                            */
  const int32_t* bloom_index;    /* int32 [num_entries]                            */
  const uint64_t* bitmask_table; /* uint64 [bitmask_rows, bitmask_words]           */
  const uint64_t* bloom_table;   /* uint64 [bloom_rows, bloom_words]               */
} grace_gtm_index;

/*
 * Request-side targeting attributes (Sec. 4.2, 4.3), one row per request.
 * Host struct of device pointers.
 */
typedef struct grace_gtm_user {
  int32_t max_locations;         /* L_max, 0..64                                   */
  int32_t reserved;              /* must be 0                                      */
  const uint64_t* bitmask;       /* uint64 [B, bitmask_words]: the user's bits     */
  const uint64_t* bloom;         /* uint64 [B, max_locations, bloom_words]: one Bloom
                                    row per user location                          */
  const int32_t* num_locations;  /* int32 [B]; clamped into [0, max_locations]     */
} grace_gtm_user;

/*
 * Decode-time constraint filter (Sec. 4, Sec. 5.4; lookup of App. A).  Beam row
 * r = b*M + m sits at trie node node_ids[r].  Token v is allowed for it when
 *   CD:  some child entry e of the node has tokens[e] = v, and for that entry
 *   GTM: (bitmask_table[bitmask_index[e]] & user.bitmask[b]) == user.bitmask[b]
 *        over all words (every user attribute bit is present), and
 *        (loc & bloom_table[bloom_index[e]]) == loc for at least one of the
 *        request's num_locations[b] location rows loc (none: not allowed).
 * Writes mask[r, w] for every word w < ceil(vocab/32): bit v % 32 of word v / 32
 * set = v allowed, the filter grace_beam_scores consumes.  A negative node id
 * is a dead beam (no token allowed).  A node id >= num_nodes, or a child entry
 * whose token or matcher ids are out of range, allows nothing for it and sets
 * *err_flag.
 *
 *   index, user   host structs (above)
 *   node_ids      device int32 [B*M]
 *   B, M          requests and beams per request; B*M*ceil(vocab/32) below 2^31
 *   mask          device uint32 [B*M, ceil(vocab/32)], written; must not overlap inputs
 *   err_flag      device int32 or NULL; set to 1 on bad index data, never cleared
 *   stream        hipStream_t
 */
int32_t grace_gtm_mask(const grace_gtm_index* index, const grace_gtm_user* user,
                       const int32_t* node_ids, int32_t B, int32_t M, uint32_t* mask,
                       int32_t* err_flag, void* stream);

/*
 * Trie step after top-k (Sec. 4.4: the selected child node ids become the next
 * step's node ids).  New beam i = b*k + j has parent p = parents[i] (request-
 * local, [0, M_prev)) and token tokens[i]:
 *   node_next[i] = child of node_prev[b*M_prev + p] reached by tokens[i],
 *                  or -1 if that parent is dead or the token is not a child
 *                  (a filtered candidate kept as a dead beam).
 * A parent outside [0, M_prev) or a node id >= num_nodes gives -1 and sets *err_flag.
 *
 *   node_prev     device int32 [B*M_prev];  parents, tokens  device int32 [B*k]
 *   node_next     device int32 [B*k], written; must not overlap the inputs
 */
int32_t grace_trie_advance(const grace_gtm_index* index, const int32_t* node_prev,
                           const int32_t* parents, const int32_t* tokens, int32_t B,
                           int32_t M_prev, int32_t k, int32_t* node_next, int32_t* err_flag,
                           void* stream);

/*
 * Graph capture (Sec. 5: the fixed-length decoding loop is captured as one
 * graph).  Every entry point above only enqueues kernels on its stream; it
 * never allocates, synchronises or sets memory, so calls made on `stream`
 * between grace_graph_begin and grace_graph_end are recorded, not run, and the
 * returned executable graph replays them all with one grace_graph_launch.
 * Pointers and sizes are frozen at capture: a replay reads and writes the same
 * buffers, which the caller keeps alive until grace_graph_destroy.
 *
 *   grace_graph_begin(stream)            start capturing on `stream` (hipStream_t,
 *                                        not NULL: the null stream cannot be
 *                                        captured); thread-local capture mode
 *   grace_graph_end(stream, &exec)       stop capturing, instantiate; *exec receives
 *                                        the executable graph (NULL on failure)
 *   grace_graph_launch(exec, stream)     replay on `stream`
 *   grace_graph_destroy(exec)            free the executable graph (NULL is a no-op)
 *   grace_graph_last_hip_error()         hipError_t of the last failed graph call
 *                                        in this thread
 * Each returns GRACE_OK, GRACE_ERR_NULL or GRACE_ERR_HIP.
 */
int32_t grace_graph_begin(void* stream);
int32_t grace_graph_end(void* stream, void** graph_exec);
int32_t grace_graph_launch(void* graph_exec, void* stream);
int32_t grace_graph_destroy(void* graph_exec);
int32_t grace_graph_last_hip_error(void);

/* Number of counters grace_debug_counts fills. */
#define GRACE_DEBUG_KINDS 8

/*
 * Device-side checks of the debug build.  The library also builds as
 * libgrace_debug.so (sources compiled with -DGRACE_DEBUG): the same entry
 * points and results, but the attention kernels (cross-attention, append,
 * self-attention, fused) count every index they had to clamp and check each
 * global row index they compute against the extent of its buffer.  This call
 * synchronises the current GPU, copies the counters to counts[0 ..
 * GRACE_DEBUG_KINDS-1] and clears them:
 *   counts[0]  request offsets out of order or outside [0, sum_L]
 *   counts[1]  parents outside [0, M_prev)
 *   counts[2]  block ids outside the pool
 *   counts[3]  computed row indices outside their buffer (an indexing error)
 *   counts[4..7] unused (0)
 * Each is a number of checking lanes or workgroups, not of distinct inputs.
 *
 *   counts   host uint32 [GRACE_DEBUG_KINDS], written (zeros on any error)
 * Returns GRACE_OK in the debug build and GRACE_ERR_UNSUPPORTED in the
 * release build (counts all zero); GRACE_ERR_NULL for a NULL counts.
 */
int32_t grace_debug_counts(uint32_t* counts);

/* Human-readable name of a status code (static storage; never NULL). */
const char* grace_status_string(int32_t status);

/* hipError_t of the last failed HIP call in this thread (0 if none). */
int32_t grace_last_hip_error(void);

/* ABI version of this header; bumped on any incompatible change. */
int32_t grace_abi_version(void);

#define GRACE_ABI_VERSION 1

#ifdef __cplusplus
}
#endif

#endif /* GRACE_H */
