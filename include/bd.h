/*
 * libbd: the BudgetDraft sparse-drafter / full-verifier hot path on MI355X (gfx950).
 *
 * Greedy speculative decoding with a drafter that reads a budgeted subset of
 * its KV cache and a verifier that reads its full cache (Sec. 3.1, Alg. 2),
 * and the continuation-block attention of multi-view training (Alg. 1).
 * Each operation is an asynchronous launch on a caller-given HIP stream:
 *
 *   bd_select_kv           budgeted KV selection (Alg. 2 "sparsify")
 *   bd_select_kv_chunks    chunk-level selection (TopKChunks, Sec. 3.4)
 *   bd_sparse_decode_attn  drafter attention over the selected entries (Eq. 2)
 *   bd_multiview_attn      a query block under several budgets + the full cache (Alg. 1)
 *   bd_multiview_attn_bwd  its gradients for the drafter's training losses (Alg. 1)
 *   bd_verify_attn         verifier attention at the gamma+1 draft positions (Eq. 1)
 *   bd_verify_attn_noalloc the same with a fixed in-library scratch (no workspace)
 *   bd_accept_len          greedy accepted-prefix length and bonus token (Eq. 3)
 *   bd_cache_append        per-round cache growth (Alg. 2)
 *   bd_cache_rollback      the accepted speculative rows kept after verification (Alg. 2)
 *   bd_top1_ce             top-1 cross-entropy against the verifier (Eqs. 5-7)
 *   bd_sample_budgets      B ~ Cat(B, w) per training sample (Alg. 1)
 *
 * Common conventions
 *   - Tensors are raw device pointers.  bf16 data are passed as uint16_t bit
 *     patterns; head_dim must be 128.
 *   - GQA: query head h reads KV head h / G, G = num_q_heads / num_kv_heads.
 *   - Positions: sequence s holds cache rows 0 .. L_s-1 (L_s = seq_lens[s]),
 *     query rows included.  A query at position p sees keys t with 0 <= t <= p.
 *     Keys and queries are post-RoPE; positions are used only for the causal rule.
 *   - Softmax scale is the caller's `scale`, positive and finite (normally
 *     1/sqrt(128)); softmax and
 *     accumulation are fp32, outputs are rounded to bf16 (nearest-even), and
 *     log-sum-exp outputs are fp32 natural logs.  A row with no visible key
 *     gets output 0 and log-sum-exp -inf.
 *   - Ownership: the caller owns every buffer; inputs are only read; outputs
 *     are overwritten in full; the library keeps no pointer after returning.
 *   - Workspace: each operation takes caller-allocated device memory of at
 *     least bd_<op>_workspace_bytes(...) bytes (256-byte aligned).  Its first
 *     BD_WS_COUNTER_BYTES hold completion counters and must be zero before the
 *     first use; every call that runs to completion leaves them zero again and
 *     writes its other scratch only past them.  One workspace can therefore
 *     serve any sequence of calls, of any operation and shape, issued on one
 *     stream.  Calls that overlap in time (two streams) must not share a
 *     workspace.  The library never allocates device memory.  A size function
 *     returns 0 for arguments its operation rejects.
 *   - Errors: arguments are checked on the host before anything is launched;
 *     on error nothing is launched and no output is touched.  A launch failure
 *     reported by the HIP runtime is BD_ERR_DEVICE.  No C++ exception crosses
 *     this interface.  bd_last_error() gives the reason of the last failure
 *     on the calling thread.  Operations on the KV cache refuse more than 2^24
 *     (sequence, KV head) pairs or more than 2^16 query heads per KV head as
 *     BD_ERR_UNSUPPORTED.
 *   - Device-side bounds: entries of idx outside [0, L_s) are skipped, counts
 *     above the stated maxima are clamped, and paged keys whose page number is
 *     outside [0, num_pages) are skipped, so malformed device data cannot make
 *     a kernel read out of bounds.
 */
#ifndef BD_H_
#define BD_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BD_ABI_VERSION 3
#define BD_HEAD_DIM 128
/* Longest candidate prefix L_s - W that bd_select_kv ranks in one pass. */
#define BD_SELECT_MAX_PREFIX 32768
/* Leading workspace bytes reserved for completion counters and other state that
 * every completed call returns to zero: one BD_WS_COUNTER_STRIDE-byte line per
 * counter, so that counters of different work units never share a cache line.
 * A call needing more than BD_WS_COUNTER_LINES lines is unsupported. */
#define BD_WS_COUNTER_BYTES 1048576
#define BD_WS_COUNTER_STRIDE 128
#define BD_WS_COUNTER_LINES (BD_WS_COUNTER_BYTES / BD_WS_COUNTER_STRIDE)

typedef int32_t bd_status;
#define BD_OK 0
#define BD_ERR_INVALID_ARG 1 /* a pointer, size or shape that the contract forbids */
#define BD_ERR_UNSUPPORTED 2 /* a valid request the library does not implement (head_dim != 128,
                               launches of 2^22 or more workgroups, ...) */
#define BD_ERR_WORKSPACE 3   /* workspace missing, too small or misaligned */
#define BD_ERR_DEVICE 4      /* the HIP runtime rejected a launch */

/* KV cache of one layer: K and V of every sequence and KV head.
 *
 * Contiguous layout (page_table == NULL): element (s, g, t, d) lives at
 *   s*stride_seq + g*stride_head + t*stride_tok + d          (elements).
 * Paged layout (page_table != NULL): element (s, g, t, d) lives at
 *   page_table[s*max_pages_per_seq + t/page_size]*stride_page
 *     + g*stride_head + (t % page_size)*stride_tok + d.
 * In both layouts d is contiguous.  K and V share the layout.  Page numbers
 * belong in [0, num_pages): no value makes a kernel read outside the pool,
 * and the attention calls treat the keys of a page numbered outside it as
 * absent (they take no weight).  A page_size that is a multiple of 16 lets
 * the verifier's full-cache pass and the selection's scoring passes read
 * through one table entry per page, which allows far longer splits per
 * workgroup than other page sizes. */
typedef struct bd_kv_desc {
  const uint16_t* k;          /* bf16 keys */
  const uint16_t* v;          /* bf16 values (ignored, may be NULL, for bd_select_kv) */
  int32_t num_seqs;           /* S >= 1 */
  int32_t num_kv_heads;       /* Hkv >= 1 */
  int32_t head_dim;           /* must be 128 */
  int32_t max_seq_len;        /* host bound: every seq_lens[s] <= max_seq_len */
  const int32_t* seq_lens;    /* device [S]: L_s, clamped to [0, max_seq_len] */
  int64_t stride_seq;         /* contiguous layout only */
  int64_t stride_head;
  int64_t stride_tok;
  const int32_t* page_table;  /* NULL, or device [S][max_pages_per_seq] page numbers */
  int32_t page_size;          /* paged: tokens per page (>= 1) */
  int32_t max_pages_per_seq;  /* paged: max_seq_len <= max_pages_per_seq * page_size */
  int32_t num_pages;          /* paged: pages in the pool */
  int64_t stride_page;        /* paged: elements between pages */
} bd_kv_desc;

const char* bd_status_string(bd_status status);
/* Reason of the last non-BD_OK status returned on this thread (static storage). */
const char* bd_last_error(void);
int32_t bd_abi_version(void);

/* ------------------------------------------------------------------------
 * bd_select_kv -- budgeted KV selection, K_S^sp(B) of Eq. (2).
 *
 * Alg. 2 sparsifies the drafter's prefix cache once after prefill; Sec. 3.4
 * keeps the entries with the largest cumulative attention weight.  For every
 * sequence s and KV head g:
 *   1. raw[t] = sum over the G query heads of g and the W observation rows i
 *      (row i at position L_s-W+i) of softmax_t(scale * <q_{h,i}, k_t>), each
 *      row normalised over its causal range t <= L_s-W+i;
 *   2. pooled[t] = max of raw over [t-r, t+r] cut to [0, N), r = pool_kernel/2,
 *      for the N = L_s - W prefix positions;
 *   3. keep the B - W prefix positions ranked first by (pooled descending,
 *      position ascending), in ascending order, then append the W window
 *      positions N .. L_s-1.
 * If B >= L_s every position 0 .. L_s-1 is kept (the sparse cache is the full
 * cache) and the scores of that sequence are not computed.
 *
 * q_win      [S][W][Hq][128] bf16: the last W query rows of each sequence.
 * lse_win    NULL, or [S][W][Hq] fp32 natural-log log-sum-exp of each window
 *            row over its causal range; when given, one pass over K suffices.
 * idx_out    [S][Hkv][budget] int32 ascending positions; slots past nsel = -1.
 * nsel_out   [S] int32: min(budget, L_s).
 * scores_out NULL, or [S][Hkv][max_seq_len] fp32 raw scores (step 1) for
 *            t < L_s of every sequence with B < L_s; other entries untouched.
 * Requirements: 1 <= window <= budget; pool_kernel odd >= 1; every
 * L_s >= window; max_seq_len - window <= BD_SELECT_MAX_PREFIX; K only (kv->v unused).
 * ---------------------------------------------------------------------- */
size_t bd_select_kv_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                    int32_t window, int32_t max_seq_len);
bd_status bd_select_kv(const bd_kv_desc* kv, const uint16_t* q_win, int32_t num_q_heads, int32_t window,
                       int32_t budget, int32_t pool_kernel, float scale, const float* lse_win,
                       int32_t* idx_out, int32_t* nsel_out, float* scores_out,
                       void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_select_kv_chunks -- chunk-level selection (TopKChunks; Sec. 3.4, Alg. 1
 * step 4, Alg. 2 "sparsify").
 *
 * Step 1 as bd_select_kv.  The prefix [0, N), N = L_s - W, is cut into chunks
 * of `chunk` positions (chunk c covers [c*chunk, min((c+1)*chunk, N)); the last
 * one is shorter when chunk does not divide N); a chunk's score is the sum of
 * its positions' raw scores (fp32, left to right).  Sec. 3.4 retains the top
 * floor(B / chunk) chunks of the prefix cache, and the W rows that scored it
 * (the continuation block of Alg. 1) attend on top of them:
 *   budget_counts_window = 0  keep floor(B / chunk) chunks, then the W window
 *                             positions: ld = B + W index slots per head;
 *   budget_counts_window = 1  B also pays for the window: floor((B - W) / chunk)
 *                             chunks, then the window; ld = B slots.
 * The kept chunks (ranked by score descending, chunk index ascending) give
 * their positions in ascending order, then the window positions N .. L_s-1.
 * idx_out    [S][Hkv][ld] int32; a head's slots past its kept positions (fewer
 *            than ld when chunk does not divide the prefix budget, or a short
 *            last chunk is kept) are -1, which the attention calls skip.
 * nsel_out   [S] int32: min(ld, L_s) (slots, not kept positions); L_s when
 *            B >= L_s, where every position is kept.
 * Other arguments, requirements and the workspace are those of bd_select_kv
 * (bd_select_kv_workspace_bytes); chunk >= 1; budget_counts_window 0 or 1.
 * ---------------------------------------------------------------------- */
bd_status bd_select_kv_chunks(const bd_kv_desc* kv, const uint16_t* q_win, int32_t num_q_heads, int32_t window,
                              int32_t budget, int32_t chunk, int32_t budget_counts_window, float scale,
                              const float* lse_win, int32_t* idx_out, int32_t* nsel_out, float* scores_out,
                              void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_sparse_decode_attn -- drafter decode attention over K_S^sp(B) (Eq. 2; Alg. 2 "draft").
 *
 * One query per head at position L_s-1 attends the entries
 * idx[s][g][0 .. nsel[s]-1] of its KV head (entries outside [0, L_s) are
 * skipped; order does not matter).
 * q       [S][Hq][128] bf16.
 * idx     [S][Hkv][ld_idx] int32; nsel [S] int32, clamped to [0, ld_idx].
 * out     [S][Hq][128] bf16; lse_out NULL or [S][Hq] fp32.
 * ---------------------------------------------------------------------- */
size_t bd_sparse_decode_attn_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                             int32_t ld_idx);
bd_status bd_sparse_decode_attn(const bd_kv_desc* kv, const uint16_t* q, int32_t num_q_heads,
                                const int32_t* idx, int32_t ld_idx, const int32_t* nsel, float scale,
                                uint16_t* out, float* lse_out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_multiview_attn -- continuation block under several sparse views and
 * the full cache (Alg. 1 steps 3 and 4).
 *
 * Row c of the block sits at position L_s - C + c.  Under view v it sees
 * {t in idx_views[v][s][g][0 .. nsel_views[v][s]-1] : t <= its position};
 * under the full branch it sees every t <= its position.
 * q_blk      [S][C][Hq][128] bf16.
 * idx_views  [V][S][Hkv][ld_idx] int32; nsel_views [V][S] int32.
 * out_views  [V][S][C][Hq][128] bf16 (may be NULL only when V == 0).
 * lse_views  NULL or [V][S][C][Hq] fp32.
 * out32_views NULL or [V][S][C][Hq][128] fp32: the outputs before rounding.
 * out_full   NULL (full branch skipped) or [S][C][Hq][128] bf16.
 * lse_full, out32_full  as for the views (ignored when out_full is NULL).
 * Training outputs: when out32_views or out32_full is given, every softmax
 * weight enters the weighted sum of values as two bf16 terms (the rounded
 * weight and its rounded remainder), so the fp32 outputs carry the weights
 * to about 2^-17 rather than 2^-9 (the bf16 outputs are then the rounding
 * of these).  bd_multiview_attn_bwd takes out32 and lse.
 * Requirements: C >= 1, V >= 0, V + (out_full != NULL) >= 1; with more than
 * 32 query rows per KV head (C * G > 32) or training outputs, at most 64
 * branches (V + (out_full != NULL)), else BD_ERR_UNSUPPORTED.
 * ---------------------------------------------------------------------- */
size_t bd_multiview_attn_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                         int32_t block_len, int32_t num_views, int32_t ld_idx,
                                         int32_t max_seq_len, int32_t with_full);
bd_status bd_multiview_attn(const bd_kv_desc* kv, const uint16_t* q_blk, int32_t num_q_heads, int32_t block_len,
                            int32_t num_views, const int32_t* idx_views, int32_t ld_idx,
                            const int32_t* nsel_views, float scale, uint16_t* out_views, float* lse_views,
                            float* out32_views, uint16_t* out_full, float* lse_full, float* out32_full,
                            void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_multiview_attn_bwd -- gradients of bd_multiview_attn for the drafter's
 * training losses (Alg. 1 steps 3-5).
 *
 * The losses reach the block's queries through every view and the full
 * branch, and its keys and values through the cache rows the block itself
 * wrote (positions L_s - C .. L_s - 1); the prefix cache is computed without
 * gradient (Alg. 1 step 2) and gets none.  With P the softmax weights of a
 * branch (from its log-sum-exp) and D_r = <dO_r, O_r>:
 *   dS = P o (dO V^T - D),  dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO,
 * summed over the branches.  A key listed m times in a view counts m times.
 * Shapes and visibility are those of bd_multiview_attn:
 * q_blk      [S][C][Hq][128] bf16; idx_views [V][S][Hkv][ld_idx]; nsel_views [V][S].
 * out32_views, lse_views  the forward's training outputs of the views (out32_views and
 *            lse_views of bd_multiview_attn: [V][S][C][Hq][128] and [V][S][C][Hq] fp32);
 *            dout_views their upstream gradients, [V][S][C][Hq][128] bf16.
 * out32_full, lse_full, dout_full  the same for the full branch: all three NULL (no
 *            full branch) or all three given.
 * D_r = <dO_r, O_r> cancels against <dO_r, v_t> where a row's weight
 * concentrates on few keys, so O enters as the fp32 training output: a bf16
 * output there would put its own rounding into every dS of the row.
 * dq         [S][C][Hq][128] fp32 (required).
 * dk_blk, dv_blk  NULL (skipped) or both [S][C][Hkv][128] fp32: row c is the
 *            gradient of cache row L_s - C + c of KV head g (0 where that position is < 0).
 * Requirements: 1 <= C <= 1024, C * G <= 1048576, V >= 0, between one and 64
 * branches (V + full), S * Hkv * (ceil(C*G/256) + 1) <= BD_WS_COUNTER_LINES.  Results do not depend on
 * scheduling (fixed summation order).
 * ---------------------------------------------------------------------- */
size_t bd_multiview_attn_bwd_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                             int32_t block_len, int32_t num_views, int32_t ld_idx,
                                             int32_t max_seq_len, int32_t with_full);
bd_status bd_multiview_attn_bwd(const bd_kv_desc* kv, const uint16_t* q_blk, int32_t num_q_heads, int32_t block_len,
                                int32_t num_views, const int32_t* idx_views, int32_t ld_idx,
                                const int32_t* nsel_views, float scale,
                                const float* out32_views, const float* lse_views, const uint16_t* dout_views,
                                const float* out32_full, const float* lse_full, const uint16_t* dout_full,
                                float* dq, float* dk_blk, float* dv_blk,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_verify_attn -- verifier attention over the full cache at the gamma+1
 * draft positions (Eq. 1; Alg. 2 "verify").
 *
 * Row j (0 .. gamma) sits at position L_s - gamma - 1 + j and sees keys
 * 0 .. that position (causal among the drafts).
 * q       [S][gamma+1][Hq][128] bf16.
 * out     [S][gamma+1][Hq][128] bf16; lse_out NULL or [S][gamma+1][Hq] fp32.
 * ---------------------------------------------------------------------- */
size_t bd_verify_attn_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t num_q_heads,
                                      int32_t gamma, int32_t max_seq_len);
bd_status bd_verify_attn(const bd_kv_desc* kv, const uint16_t* q, int32_t num_q_heads, int32_t gamma, float scale,
                         uint16_t* out, float* lse_out,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_verify_attn_noalloc -- bd_verify_attn without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).
 *
 * Same operation, arguments, kernels and results (bit for bit) as
 * bd_verify_attn.  Its scratch (completion counters, then split records) is a
 * fixed array of BD_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held
 * until the process ends; nothing is allocated by this call or by the library.
 * The first call on a device resolves the array's address and clears its counter
 * region with one small kernel on `stream`.  Every call on a GPU shares that
 * GPU's array: calls that overlap in time on one GPU (other streams, other host
 * threads) race and must not be issued.  A shape whose plan needs more scratch
 * than the fixed size returns BD_ERR_UNSUPPORTED before anything is launched
 * (the 16K batch of 8 sequences, contiguous or paged, fits).
 * ---------------------------------------------------------------------- */
#define BD_NOALLOC_SCRATCH_BYTES 16777216
bd_status bd_verify_attn_noalloc(const bd_kv_desc* kv, const uint16_t* q, int32_t num_q_heads, int32_t gamma,
                                 float scale, uint16_t* out, float* lse_out, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_accept_len -- greedy acceptance (Eq. 3; Alg. 2 accept + bonus token).
 *
 * a*_i = lowest index among the maxima of logits row i (i = 0 .. gamma;
 * -0.0 equals +0.0).  Row i is the verifier's prediction for draft i.
 * accept = largest k <= gamma with draft[i] == a*_i for every i < k;
 * bonus = a*_k.
 * logits  row (s, i) at logits + (s*(gamma+1) + i) * row_stride, fp32, finite.
 * draft   [S][gamma] int32.
 * accept_out [S] int32; bonus_out NULL or [S]; argmax_out NULL or [S][gamma+1].
 * Requirements: gamma >= 0, vocab >= 1, row_stride >= vocab.  BD_ERR_UNSUPPORTED
 * for gamma > 63 and for shapes whose launch would exceed 2^22 - 1 workgroups
 * (S*(gamma+1)*ceil(vocab/8192) and more).
 * ---------------------------------------------------------------------- */
size_t bd_accept_len_workspace_bytes(int32_t num_seqs, int32_t gamma, int32_t vocab);
bd_status bd_accept_len(const float* logits, int64_t row_stride, const int32_t* draft, int32_t num_seqs,
                        int32_t gamma, int32_t vocab, int32_t* accept_out, int32_t* bonus_out,
                        int32_t* argmax_out, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_cache_append -- append rows to a cache (Alg. 2: the caches are updated
 * with the appended tokens; during drafting the sparse cache grows by each
 * drafted token).
 *
 * For every sequence s, the n new rows go to positions L_s .. L_s+n-1, where
 * L_s = kv->seq_lens[s]; rows at or past kv->max_seq_len (the capacity) are
 * dropped.  kv->k and kv->v are written (the descriptor's pointers must be
 * writable), and kv->seq_lens (device) is advanced in place by the rows written.
 * k_new, v_new [S][n][Hkv][128] bf16, 16-byte aligned.
 * idx, nsel  NULL, or the drafter's sparse list [S][Hkv][ld_idx] and count [S]
 *            (device, updated in place): every written position is appended to
 *            each head's list at slots nsel[s] ..; slots past ld_idx are dropped.
 * Two launches on `stream` (row copies, then the counts).  Contiguous or paged
 * layouts (paged: the pages of the new positions must already be mapped).
 * ---------------------------------------------------------------------- */
bd_status bd_cache_append(const bd_kv_desc* kv, const uint16_t* k_new, const uint16_t* v_new, int32_t n,
                          int32_t* idx, int32_t ld_idx, int32_t* nsel, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_cache_rollback -- keep the accepted speculative rows after verification
 * (Alg. 2, cache update after the accept step).
 *
 * Each sequence's last `spec` rows are speculative and the first accept[s] of
 * them (clamped to [0, spec]) were accepted.
 *   base_lens given (the lengths before this round's speculative appends, e.g. a
 *     device copy of seq_lens taken before them): seq_lens[s] = min(seq_lens[s],
 *     base_lens[s] + accept[s]); with base_nsel likewise nsel[s] = min(nsel[s],
 *     base_nsel[s] + accept[s]).  Rows an append dropped at the capacity, and
 *     list entries it dropped past ld_idx, were never counted, so an accepted row
 *     stays only if it was written and no committed row or entry is removed.
 *   base_lens / base_nsel NULL: spec - accept[s] is subtracted (never below 0),
 *     which is right only when every speculative row and list entry was written.
 * seq_lens, nsel: device int32 [S], updated in place (nsel may be NULL; base_nsel
 * needs nsel); accept: device [S] (e.g. bd_accept_len's accept_out); base_lens,
 * base_nsel: NULL or device [S].  One launch on `stream`.
 * ---------------------------------------------------------------------- */
bd_status bd_cache_rollback(int32_t* seq_lens, int32_t* nsel, const int32_t* accept, int32_t num_seqs, int32_t spec,
                            const int32_t* base_lens, const int32_t* base_nsel, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_top1_ce -- top-1 cross-entropy of the drafter against the verifier's
 * greedy targets: the target of row r is the lowest-index argmax of the
 * verifier's logits (Eq. 5), and loss[r] = logsumexp(student[r]) -
 * student[r][target] (natural log) is the row's summand of L_A (Eq. 6, full
 * cache) or L_C (Eq. 7, sparse cache).  The targets' scan and the loss share
 * one pass over the two logit rows.
 *
 * student     [rows][vocab] fp32, rows student_stride elements apart.
 * teacher     NULL, or [rows][vocab] fp32 verifier logits (teacher_stride):
 *             the targets are their argmax.
 * targets     used when teacher is NULL: [rows] int32; an entry outside
 *             [0, vocab) gives loss NaN and target -1.
 * loss_out    [rows] fp32; target_out NULL or [rows] int32; lse_out NULL or
 *             [rows] fp32 (logsumexp of the student row).
 * Exactly one of teacher and targets; rows <= BD_WS_COUNTER_LINES.
 * ---------------------------------------------------------------------- */
size_t bd_top1_ce_workspace_bytes(int32_t rows, int32_t vocab);
bd_status bd_top1_ce(const float* student, int64_t student_stride, const float* teacher, int64_t teacher_stride,
                     const int32_t* targets, int32_t rows, int32_t vocab, float* loss_out, int32_t* target_out,
                     float* lse_out, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bd_sample_budgets -- B ~ Cat(budgets, weights), one draw per uniform number
 * (Sec. 3.4 and Alg. 1 step 4 draw the training budget this way).
 *
 * Thresholds t_j = (w_0 + ... + w_j) / (w_0 + ... + w_{n-1}) are formed on the
 * host in fp32 (sums in order, then one division each); out[i] = budgets[j]
 * for the first j with u[i] < t_j (the last budget if none).  The random
 * numbers are the caller's: u [count] fp32 in [0, 1) on the device.
 * budgets, weights: host arrays of n <= 16 entries, weights positive and finite.
 * out [count] int32 on the device.
 * ---------------------------------------------------------------------- */
bd_status bd_sample_budgets(const float* u, int32_t count, const int32_t* budgets, const float* weights, int32_t n,
                            int32_t* out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* BD_H_ */
