/*
 * pd.h -- C ABI of the MI355X (gfx950) block-sparse attention path of
 * Prefilling-dLLM: chunked prefill, per-step chunk/token selection, and
 * sparse decode attention.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Plain C.  No HIP or torch types: device buffers are `void *` (or typed
 *   pointers to device memory), the stream is a `hipStream_t` passed as
 *   `void *` (NULL = the default stream).
 * - Ownership: every pointer is caller-owned DEVICE memory, contiguous in the
 *   layout stated next to it, 16-byte aligned.  The library allocates nothing,
 *   frees nothing and never synchronises; every call only enqueues kernels on
 *   `stream` and returns.  Scratch space is the caller's `workspace`, sized by
 *   pd_workspace_bytes().  Calls on different streams must not share outputs
 *   or workspace.
 * - Errors: arguments are checked on the host before anything is launched; on
 *   error nothing is launched, no output is touched, a status is returned and
 *   a thread-local message is kept for pd_last_error_message().  A failed
 *   launch returns PD_ERR_HIP.  Faults inside a kernel surface at the caller's
 *   next synchronisation on `stream`.
 * - Size limits besides those of each entry point: element offsets inside one
 *   sequence's cache, chunk sequence, decode block or decode KV rows stay
 *   below 2^31, and every launch grid (prefill, selection, decode, Split-S
 *   merge) below 2^31 workgroups; larger calls return PD_ERR_BAD_DIMS, and
 *   the size queries return 0 for them.
 * - Element type: all Q/K/V/O/cache tensors of one call have the type
 *   `dims->dtype` (bf16 or fp32).  Scores, key means and LSEs are fp32;
 *   indices are int32.  Arithmetic is fp32 (bf16 inputs feed bf16 matrix
 *   cores with fp32 accumulation; the attention probabilities are rounded to
 *   bf16 before the P*V product on the bf16 path and stay fp32 on the fp32
 *   path).
 *
 * Symbols (the paper's problem statement, Section 5): B sequences, N chunks of
 * C content tokens each with a BOS token prepended, L_q query rows, L_m (= |m|)
 * pseudo-label rows, L_d decode rows, H_q query heads, H_kv key/value heads
 * (query head h reads KV head h / (H_q/H_kv)), head dimension d, top-K chunks
 * and a budget of B_tok tokens per kept chunk.  S_c = 1 + C + L_q + L_m is the
 * length of one chunk sequence [BOS; c; q; m].
 */
#ifndef PD_H
#define PD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PD_OK = 0,
  PD_ERR_NULL_PTR = 1,    /* a required pointer is NULL                          */
  PD_ERR_BAD_DIMS = 2,    /* a size is out of range (see each entry point)       */
  PD_ERR_UNSUPPORTED = 3, /* H_q % H_kv != 0, d not in {64,128}, unknown dtype    */
  PD_ERR_MISALIGNED = 4,  /* a pointer is not 16-byte aligned                     */
  PD_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than pd_workspace_bytes()  */
  PD_ERR_HIP = 6          /* a kernel launch failed                               */
} pd_status;

typedef enum { PD_BF16 = 0, PD_FP32 = 1 } pd_dtype;

typedef struct {
  int32_t batch;        /* B >= 1                                                   */
  int32_t n_chunks;     /* N, 1..1024                                               */
  int32_t chunk_len;    /* C, 1..4096 content tokens; the cache holds 1+C rows      */
  int32_t q_len;        /* L_q >= 1 query rows                                      */
  int32_t m_len;        /* L_m >= 0 pseudo-label rows                               */
  int32_t dec_len;      /* L_d >= 1 decode rows                                     */
  int32_t n_heads_q;    /* H_q >= 1                                                 */
  int32_t n_heads_kv;   /* H_kv >= 1, divides H_q                                   */
  int32_t head_dim;     /* d, 64 or 128                                             */
  int32_t dtype;        /* pd_dtype                                                 */
  float sm_scale;       /* softmax scale; <= 0 selects 1/sqrt(d)                    */
  int32_t qm_per_chunk; /* 0: the q/m rows are one tensor shared by all chunks,
                           [B][L_q+L_m][H][d];  1: one copy per chunk,
                           [B][N][L_q+L_m][H][d]                                    */
  int32_t out_fp32;     /* 0: o and o_dec have element type dtype; 1: they are fp32
                           (bf16 inputs, fp32 outputs: no output rounding)          */
  int32_t tok_score_dir; /* token score of pd_prefill_chunks: 0 = both sums of
                           Eq. 5 (default); 1 = its first sum only, the mass the
                           query rows put on the token (the query-to-chunk score
                           of the paper's retention-score ablation)                 */
} pd_dims;

/*
 * Stage (a), one layer: chunk prefill (Section 5.1, Eq. 2), the chunk KV
 * cache, the chunk key summary, and the eviction score of Eq. 5 (Section 5.2).
 *
 * For every sequence b, chunk n and query head h, the S_c rows
 * [BOS; c_1..c_C; q_1..q_Lq; m_1..m_Lm] of chunk n attend to each other with
 * full bidirectional softmax(scale * Q K^T) V and to nothing outside the chunk.
 *
 * Inputs (element type dims->dtype):
 *   q_pre  [B][N][1+C][H_q][d]   chunk rows, slot 0 = the BOS token
 *   k_pre, v_pre [B][N][1+C][H_kv][d]
 *   q_qm   query + pseudo-label rows, [B][L_q+L_m][H_q][d] (shared) or
 *          [B][N][L_q+L_m][H_q][d] (qm_per_chunk = 1); rows 0..L_q-1 are the
 *          query rows
 *   k_qm, v_qm  likewise with H_kv heads
 * Outputs:
 *   o         [B][N][S_c][H_q][d]   attention output, rows ordered BOS, c, q, m
 *             (element type dtype, or fp32 when out_fp32 = 1)
 *   k_cache, v_cache [B][N][H_kv][1+C][d]  exact copies of the chunk rows
 *             (BOS at slot 0), chunk-contiguous per KV head
 *   tok_score fp32 [B][N][C]  e(c_j) of Eq. 5: for content token j, the
 *             softmax mass the L_q query rows put on it plus the mass it puts
 *             on the L_q query columns, summed over all H_q heads (the first
 *             term alone when dims->tok_score_dir = 1)
 *   tok_rank  int32 [B][N][C]  rank of token j among the C tokens of its chunk
 *             by tok_score: 0 = highest, ties to the lower index (Section 5.2:
 *             tokens are ranked by eviction score)
 *   key_mean  fp32 [B][N][H_kv][d]  mean of the C content keys (BOS excluded)
 *   chunk_score fp32 [B][N] or NULL  prefill-time chunk score, lower = more
 *             relevant: an attention-space reading of the length-normalised
 *             NLLs s_I + s_P of Section 5.1 (Eqs. 3-4).  With a(r) the mass
 *             q/m row r puts on the chunk's C content columns, averaged over
 *             the H_q heads: s = -(1/L_q) sum_{query rows} ln a(r)
 *             - (1/L_m) sum_{pseudo-label rows} ln a(r) (second term only when
 *             L_m >= 1).  Select with pd_select_ranked(lowest = 1).
 * workspace: >= pd_workspace_bytes(dims, 0, 0, 0, 0) bytes.
 * Errors: PD_ERR_BAD_DIMS for a size out of range; see the status list.
 */
pd_status pd_prefill_chunks(const pd_dims *dims,
                            const void *q_pre, const void *k_pre, const void *v_pre,
                            const void *q_qm, const void *k_qm, const void *v_qm,
                            void *o, void *k_cache, void *v_cache,
                            float *tok_score, int32_t *tok_rank, float *key_mean, float *chunk_score,
                            void *workspace, size_t ws_bytes, void *stream);

/*
 * Stage (b) from given chunk scores (Section 5.2, inter-chunk sparsity: keep
 * the K chunks with the lowest combined score), e.g. the chunk_score of
 * pd_prefill_chunks, selected once before the denoising loop.
 * Keeps the top_k lowest (lowest = 1) or highest (lowest = 0) of
 * chunk_score fp32 [B][N] (ties to the lower index; -0 equals +0), and the
 * tokens of each kept chunk with rank < tok_budget in tok_rank int32
 * [B][N][C].  Outputs as pd_score_select: chunk_idx int32 [B][top_k]
 * ascending; tok_slot int32 [B][top_k][tok_budget] ascending slots in 1..C.
 * Sizes: 1 <= top_k <= N, 1 <= tok_budget <= C.  No workspace.
 */
pd_status pd_select_ranked(const pd_dims *dims, int32_t top_k, int32_t tok_budget, const float *chunk_score,
                           int32_t lowest, const int32_t *tok_rank, int32_t *chunk_idx, int32_t *tok_slot,
                           void *stream);

/*
 * Stage (b), one layer, one denoising step: chunk scores, top-K chunks
 * (Section 5.2, inter-chunk sparsity) and the top-B_tok tokens of each kept
 * chunk by the Eq. 5 score (intra-chunk sparsity), read from the token ranks
 * that pd_prefill_chunks wrote (a token is kept iff its rank < B_tok).
 *
 * The chunk score is an attention-space stand-in for the paper's NLL score:
 *   s[b][n] = sum_h scale * < mean_r q_dec[b][r][h], key_mean[b][n][h/G] >,
 * higher = kept.  Ties rank the lower chunk (token) index first.
 * Inputs:  q_dec [B][L_d][H_q][d] (dims->dtype), key_mean fp32 [B][N][H_kv][d],
 *          tok_rank int32 [B][N][C] (a permutation of 0..C-1 per chunk).
 * Outputs: chunk_idx int32 [B][top_k], ascending chunk indices;
 *          tok_slot  int32 [B][top_k][tok_budget], ascending cache slots in
 *          1..C of the kept tokens of chunk chunk_idx[b][k] (slot = token+1);
 *          chunk_score fp32 [B][N] or NULL.
 * Sizes: 1 <= top_k <= N, 1 <= tok_budget <= C.
 * workspace: >= pd_workspace_bytes(dims, top_k, tok_budget, 0, 1) bytes.
 */
pd_status pd_score_select(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                          const void *q_dec, const float *key_mean, const int32_t *tok_rank,
                          int32_t *chunk_idx, int32_t *tok_slot, float *chunk_score,
                          void *workspace, size_t ws_bytes, void *stream);

/*
 * pd_score_select without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, outputs and errors as
 * pd_score_select minus the workspace: its scratch (the B*N*H_q*ceil(L_d/128)
 * fp32 chunk-score terms, rounded up to 256 bytes) lives in a static array of
 * 4 MiB per GPU, held by the library from the first call on that GPU until the
 * process ends; a call that needs more returns PD_ERR_BAD_DIMS.  The current device's array is used (call
 * with the stream's device current).  Every call on one GPU shares that
 * array: calls that overlap in time on one GPU (other streams, other threads)
 * race and must be serialised by the caller.  Nothing is allocated and nothing
 * needs clearing: every call rewrites the terms before it reads them.
 */
pd_status pd_score_select_noalloc(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                                  const void *q_dec, const float *key_mean, const int32_t *tok_rank,
                                  int32_t *chunk_idx, int32_t *tok_slot, float *chunk_score, void *stream);

/*
 * Stage (c), one layer, one denoising step: the L_d decode rows attend
 * (bidirectionally) over, in order, for each kept chunk chunk_idx[b][k]: its
 * BOS row (cache slot 0) and the rows at slots tok_slot[b][k][*]; then rows
 * 0..n_static-1 of the static query KV; then their own L_d rows (Section 5.3,
 * prefix reuse).  L_kv = top_k*(1+tok_budget) + n_static + L_d rows.
 *
 * Inputs (dims->dtype): q_dec [B][L_d][H_q][d]; k_dec, v_dec [B][L_d][H_kv][d];
 *   k_cache, v_cache as written by pd_prefill_chunks; k_static, v_static
 *   [B][L_q+L_m][H_kv][d] (rows 0..n_static-1 used; may be NULL when
 *   n_static = 0); chunk_idx, tok_slot as written by pd_score_select (entries
 *   must lie in 0..N-1 and 1..C).
 * Outputs: o_dec [B][L_d][H_q][d] (dtype, or fp32 when out_fp32 = 1);
 *   lse_dec fp32 [B][H_q][L_d] natural-log
 *   row LSE, or NULL (bf16 path: the log of the sum of
 *   the bf16-rounded softmax weights that multiply V, within log(1 + 2^-8)).
 * num_splits: the KV rows are cut into that many shards processed in
 *   parallel and merged by log-sum-exp (the paper's Split-S); 0 = chosen by the
 *   library from the sizes; otherwise 1..64.
 * Sizes: 1 <= top_k <= N, 1 <= tok_budget <= C, 0 <= n_static <= L_q + L_m.
 * workspace: >= pd_workspace_bytes(dims, top_k, tok_budget, num_splits, 2)
 *   bytes (may be 0, then workspace may be NULL).
 */
pd_status pd_sparse_decode_attn(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                                const void *q_dec, const void *k_dec, const void *v_dec,
                                const void *k_cache, const void *v_cache,
                                const int32_t *chunk_idx, const int32_t *tok_slot,
                                const void *k_static, const void *v_static, int32_t n_static,
                                void *o_dec, float *lse_dec, int32_t num_splits,
                                void *workspace, size_t ws_bytes, void *stream);

/*
 * Static-selection mode (the paper selects once, before the denoising loop:
 * Section 5.2 selection from the pseudo-label rows, reused for every step of
 * Section 5.3).  Three calls per layer replace the per-step pd_score_select +
 * gathered decode:
 *
 * pd_score_select_static: as pd_score_select, but the mean query is taken
 *   over the L_m pseudo-label rows of q_qm (rows L_q..L_q+L_m-1 of each
 *   sequence's q/m block, in the layout dims->qm_per_chunk gives; chunk 0's
 *   copy when per chunk) instead of the decode rows.  Needs m_len >= 1.
 *   workspace: >= pd_workspace_bytes(dims, top_k, tok_budget, 0, 1) bytes.
 *
 * pd_gather_selected: copies, once, the prefix rows a decode step reads into
 *   contiguous buffers k_sel, v_sel [B][H_kv][top_k*(1+tok_budget)][d]
 *   (dims->dtype): for each kept chunk chunk_idx[b][k] in order, its BOS row
 *   (slot 0) and then the rows at slots tok_slot[b][k][*].  Bit-exact copies;
 *   no workspace.
 *
 * pd_sparse_decode_attn_compact: pd_sparse_decode_attn whose prefix rows are
 *   rows 0..n_sel-1 of k_sel, v_sel [B][H_kv][n_sel][d] instead of rows
 *   gathered from the chunk cache (0 <= n_sel <= 2^20; k_sel/v_sel may be
 *   NULL when n_sel = 0).  With the buffers of pd_gather_selected and
 *   n_sel = top_k*(1+tok_budget) the result is that of pd_sparse_decode_attn
 *   with the same selection.  workspace: >= pd_compact_workspace_bytes bytes.
 * Errors as for the per-step calls.
 */
pd_status pd_score_select_static(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                                 const void *q_qm, const float *key_mean, const int32_t *tok_rank,
                                 int32_t *chunk_idx, int32_t *tok_slot, float *chunk_score,
                                 void *workspace, size_t ws_bytes, void *stream);
pd_status pd_gather_selected(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                             const void *k_cache, const void *v_cache,
                             const int32_t *chunk_idx, const int32_t *tok_slot,
                             void *k_sel, void *v_sel, void *stream);
pd_status pd_sparse_decode_attn_compact(const pd_dims *dims, int32_t n_sel,
                                        const void *q_dec, const void *k_dec, const void *v_dec,
                                        const void *k_sel, const void *v_sel,
                                        const void *k_static, const void *v_static, int32_t n_static,
                                        void *o_dec, float *lse_dec, int32_t num_splits,
                                        void *workspace, size_t ws_bytes, void *stream);
size_t pd_compact_workspace_bytes(const pd_dims *dims, int32_t n_sel, int32_t num_splits);

/*
 * Full-mask cache construction (Section 6, the ablation of the KV cache
 * construction strategy): once the chunks are selected, the kept rows and the
 * query are re-encoded jointly, with the decoding mask, at continuous
 * positions.  pd_gather_joint builds the joint rows of every sequence; one
 * pd_sparse_decode_attn_compact call over them (dims->dec_len = L_j,
 * n_sel = 0, n_static = 0, k_sel / v_sel / k_static / v_static NULL, q_dec,
 * k_dec, v_dec = q_joint, k_joint, v_joint) is the dense joint attention, and
 * k_pref, v_pref (the same K, V rows in the compact prefix layout) then serve
 * as the prefix (n_sel = L_j) of the decoding steps'
 * pd_sparse_decode_attn_compact calls.
 *
 * Joint rows, L_j = top_k*(1+tok_budget) + L_q per sequence: for each kept
 * chunk k = 0..top_k-1 (chunk_idx[b][k]) its BOS row (slot 0) and the rows at
 * slots tok_slot[b][k][*]; then query rows 0..L_q-1 of the q/m block (layout
 * per dims->qm_per_chunk, chunk 0's copy when per chunk).  Q rows come from
 * q_pre, K and V rows from k_cache / v_cache (kept rows) or q_qm / k_qm / v_qm
 * (query rows).
 * Positions: the chunk forward placed slot s of every chunk at s and query row
 * j at C+1+j; jointly, kept chunk k starts at k*(C+1), so its rows move by
 * k*(C+1), and the query rows move by (top_k-1)*(C+1).  Q and K are rotated
 * by the rotate-half rotary embedding with frequencies
 * rope_base^(-2i/d), i = 0..d/2-1 (element i pairs with element i + d/2);
 * the angle and the rotation are evaluated in double precision and rounded
 * once to dims->dtype.  V is copied.  rope_base = 0: no rotation (bit-exact
 * copies).
 *
 * Inputs (dims->dtype): q_pre [B][N][1+C][H_q][d] (as given to
 *   pd_prefill_chunks); k_cache, v_cache as written by pd_prefill_chunks;
 *   q_qm, k_qm, v_qm as given to pd_prefill_chunks; chunk_idx [B][top_k],
 *   tok_slot [B][top_k][tok_budget] as written by the selection calls
 *   (entries must lie in 0..N-1 and 1..C).
 * Outputs (dims->dtype, caller-owned): q_joint [B][L_j][H_q][d], k_joint and
 *   v_joint [B][L_j][H_kv][d]; k_pref and v_pref [B][H_kv][L_j][d], the same
 *   K and V values (both NULL: not written; one NULL: PD_ERR_NULL_PTR).  No
 *   workspace; asynchronous on stream.
 * Sizes: 1 <= top_k <= N, 1 <= tok_budget <= C, rope_base finite and >= 0.
 * Errors: PD_ERR_NULL_PTR, PD_ERR_MISALIGNED, PD_ERR_BAD_DIMS,
 *   PD_ERR_UNSUPPORTED, PD_ERR_HIP.
 */
pd_status pd_gather_joint(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                          const int32_t *chunk_idx, const int32_t *tok_slot,
                          const void *q_pre, const void *k_cache, const void *v_cache,
                          const void *q_qm, const void *k_qm, const void *v_qm, double rope_base,
                          void *q_joint, void *k_joint, void *v_joint, void *k_pref, void *v_pref,
                          void *stream);

/* Bytes of ONE of k_cache / v_cache for one layer: B*N*H_kv*(1+C)*d*elem. */
size_t pd_cache_bytes(const pd_dims *dims);

/* Workspace bytes for `which` = 0 prefill, 1 select, 2 decode (num_splits as
 * passed to pd_sparse_decode_attn; 0 = automatic).  Returns 0 for invalid
 * dims (the matching entry point then reports the error). */
size_t pd_workspace_bytes(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                          int32_t num_splits, int32_t which);

/* The number of KV shards pd_sparse_decode_attn uses for these arguments. */
int32_t pd_decode_splits(const pd_dims *dims, int32_t top_k, int32_t tok_budget,
                         int32_t n_static, int32_t num_splits);

/* Diagnostic: the device's achievable dense bf16 MFMA rate, the yardstick the
 * attention kernels are compared with besides the published peak.
 * Launches n_workgroups (1..2^20) workgroups of 4 waves; each wave runs iters
 * iterations of 8 v_mfma_f32_32x32x16_bf16 (32768 FLOP each) on register
 * operands, so one call performs n_workgroups * 4 * iters * 8 * 32768 FLOP.
 * sink: caller-owned device buffer of n_workgroups * 256 floats (16-B aligned)
 * that receives one value per thread.  Asynchronous on stream; time it with
 * events.  Errors: PD_ERR_NULL_PTR, PD_ERR_BAD_DIMS, PD_ERR_MISALIGNED,
 * PD_ERR_HIP. */
pd_status pd_mfma_rate_probe(int32_t n_workgroups, int32_t iters, float *sink, void *stream);

const char *pd_status_string(pd_status s);
const char *pd_last_error_message(void); /* thread-local detail of the last error */
const char *pd_version(void);

#ifdef __cplusplus
}
#endif
#endif /* PD_H */
