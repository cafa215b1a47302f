/* ubt.h -- C ABI of libubt.so: UBTree draft-tree construction on AMD Instinct MI355X
 * (gfx950).  UBTree is arXiv 2609.39972; section, equation and algorithm names below
 * refer to that paper.
 *
 * One draft step turns the proposer logits of B independent sequences into B draft
 * trees.  Sequence b carries gamma = L - 1 logit rows (draft depths 1..gamma; the block
 * of L positions includes the anchor x_0).  The calls run in this order:
 *
 *   ubt_topk           per row: softmax statistics and the top-K candidate set C_i
 *   ubt_lm_head_topk   the same from hidden states and the LM head, logits kept on chip
 *   ubt_bigram_scores  per (b, depth): selector scores Delta_i and normalised log q^bi
 *   ubt_build_tree     per sequence: beam search + global pruning -> tree and mask
 *   ubt_tree_mask      (optional) the ancestor mask of any parent-pointer tree
 *
 * and the tree is then verified by the target model:
 *
 *   ubt_tree_attention every node attends to the committed context and its ancestors
 *   ubt_verify_accept  the accepted path and the bonus token
 *   ubt_commit_kv      the accepted path's keys and values appended to the cache
 *
 * Training uses
 *
 *   ubt_tree_kl_loss   the renormalised-KL objective and its gradients
 *
 * ubt_draft_tree does ubt_bigram_scores + ubt_build_tree in one call (one launch for
 * the common shapes); ubt_draft_step the whole step.  ubt_edge_scores and
 * ubt_build_tree_best_first replace the last two calls under the unigram-plus-bigram
 * scoring (cumulative unnormalised scores, best-first growth).
 *
 * Conventions shared by every call:
 *   - Every pointer is device memory unless marked [host].  The caller owns every
 *     buffer; the library never allocates or frees device memory.
 *   - Calls are asynchronous on `stream` (a hipStream_t; 0 = the null stream).  The
 *     library never synchronises and keeps no mutable global state, so calls may be
 *     issued from several host threads and captured into HIP graphs.
 *   - Every argument check runs on the host before any launch.  On an error status
 *     nothing is launched and no output is written.  Values inside device buffers
 *     (logits, ids, scores) are not checked; the documented value ranges are the
 *     caller's responsibility, and values outside them give unspecified results but
 *     never out-of-bounds accesses.
 *   - Arrays are row-major and contiguous unless a stride is given.  Outputs sized
 *     [B, gamma, K] etc. are indexed [b][i][k] with i = 0..gamma-1 the position (draft
 *     depth i+1).
 */
#ifndef UBT_H
#define UBT_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define UBT_ABI_VERSION 1

/* Limits checked by the host-side validation. */
#define UBT_MAX_K 64          /* candidates per position */
#define UBT_MAX_GAMMA 64      /* logit rows (draft depths) per sequence */
#define UBT_MAX_BUDGET 255    /* non-root nodes per tree; N = budget + 1 <= 256 slots */
#define UBT_MAX_WIDTH 255     /* search width W */
#define UBT_MAX_EXPANSION 4096 /* W * K extensions per depth, and gamma * W supertree nodes */
#define UBT_MAX_RANK 512      /* selector rank r (a multiple of 16) */

typedef enum ubt_dtype { UBT_F32 = 0, UBT_BF16 = 1 } ubt_dtype_t;

typedef enum ubt_status {
  UBT_OK = 0,
  UBT_ERR_NULL = 1,        /* a required pointer is NULL */
  UBT_ERR_SHAPE = 2,       /* a size, stride or limit is violated */
  UBT_ERR_VALUE = 3,       /* a scalar argument is out of range (zeta > 0, alpha <= 0, ...) */
  UBT_ERR_UNSUPPORTED = 4, /* a valid combination this build does not handle */
  UBT_ERR_WORKSPACE = 5,   /* a required workspace is missing, too small or misaligned */
  UBT_ERR_HIP = 6          /* a HIP launch failed; see ubt_last_hip_error() */
} ubt_status_t;

/* Human-readable name of a status code (static storage). */
const char* ubt_status_str(ubt_status_t status);

/* UBT_ABI_VERSION of the loaded library. */
int ubt_abi_version(void);

/* hipError_t of the last launch that returned UBT_ERR_HIP on the calling host thread. */
int ubt_last_hip_error(void);

/* ------------------------------------------------------------------------------------
 * ubt_topk -- softmax statistics and candidate sets.
 * Method / Unigram Proposer, Eq. (ubtree-unigram): q_i = softmax(u_i) over the whole
 * vocabulary; "Candidate Sets": C_i = the K tokens of largest q_i.  Softmax is
 * increasing, so C_i is ranked on the logits themselves.
 *
 * logits   : u[b][i][v] at element offset b*stride_b + i*stride_i + v, dtype `dt`
 *            (UBT_BF16 or UBT_F32); values finite or -inf, at least one finite value
 *            per row; NaN gives unspecified results.  stride_i >= V, stride_b >=
 *            gamma*stride_i.  Rows whose start is 16-byte aligned take the fast path.
 * B, gamma : sequences and rows per sequence, 1 <= gamma <= UBT_MAX_GAMMA, B >= 1.
 * V        : vocabulary size, K <= V, V * sizeof(element) < 2^32 bytes.
 * K        : candidates per row, 1 <= K <= UBT_MAX_K.
 * cand_ids : int32 [B, gamma, K]   token ids ordered by (logit desc, id asc); -0 == +0.
 * cand_logit : float [B, gamma, K] the candidates' logits (exact for both dtypes).
 * cand_logprob : float [B, gamma, K] log q_i(candidate) = logit - lse; may be NULL.
 * lse      : float [B, gamma]      log sum_v exp(u_v) (natural log); may be NULL.
 * No scratch memory is used: one workgroup handles one row end to end.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_topk(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V,
                      int64_t stride_b, int64_t stride_i, int K, int32_t* cand_ids,
                      float* cand_logit, float* cand_logprob, float* lse, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_lm_head_topk -- the LM-head projection followed by ubt_topk's outputs, without
 * writing the logits.  Background, "DFlash & DFlash 2": the proposer's hidden state h_i
 * is mapped to its logits by the frozen target LM head, u_i = W_lm h_i.  Method /
 * Unigram Proposer, Eq. (ubtree-unigram) and "Candidate Sets": LSE_i and C_i as for
 * ubt_topk.
 *
 * h        : bf16 [M, d] row-major, the hidden states (M = rows over all sequences and
 *            positions, e.g. B * gamma), 16-byte aligned.
 * w_lm     : bf16 [V, d] row-major, the LM head (one row per token), 16-byte aligned.
 * M, d, V  : M >= 1; d % 32 == 0, 32 <= d <= 65536; K <= V < 2^31.
 * K        : candidates per row, 1 <= K <= UBT_MAX_K.
 * cand_ids : int32 [M, K]  token ids ordered by (logit desc, id asc).
 * cand_logit : float [M, K] the candidates' logits, fp32 sums of the exact bf16
 *            products (accumulation order unspecified).
 * cand_logprob : float [M, K] logit - lse; may be NULL.   lse : float [M]; may be NULL.
 * workspace, ws_bytes : device scratch of at least ubt_lm_head_topk_workspace_bytes(M, d,
 *            V, K) bytes, 256-byte aligned, owned by the caller; no state is kept in it
 *            between calls, and calls that share it must not overlap.
 * The head is read once per 16 rows of h (rows are taken 16 at a time); each pass is
 * bound by the bandwidth of reading w_lm.  Inputs must be finite; non-finite logits
 * give unspecified candidates.  Returns UBT_ERR_WORKSPACE for a missing, small or
 * misaligned workspace, UBT_ERR_UNSUPPORTED for shapes the workspace query rejects
 * (it returns 0 for them: very large V at large K).
 * ------------------------------------------------------------------------------------ */
size_t ubt_lm_head_topk_workspace_bytes(int M, int d, int64_t V, int K);
ubt_status_t ubt_lm_head_topk(const void* h, const void* w_lm, int M, int d, int64_t V, int K,
                              int32_t* cand_ids, float* cand_logit, float* cand_logprob,
                              float* lse, void* workspace, size_t ws_bytes,
                              hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_bigram_scores -- selector scores and normalised transition log-probabilities.
 * Background, Eq. (dflash2-selector): delta_i(a, b) = (P(h_i) (.) phi(a))^T psi(b).
 * Method / Parallel Computation, Eq. (ubtree-edge-matrix): Delta_i = Phi_{i-1}
 * diag(P(h_i)) Psi_i^T over all pairs of C_{i-1} x C_i, with C_0 = {x_0}.
 * Method / Depth Calibration, Eq. (ubtree-depth): s_i = alpha_i u_i(b) + lambda_i delta_i.
 * Appendix A / Path Scores, Eq. (ubtree-path): log q_i^bi(b|a) = s_i(a,b) -
 * log sum_{v in C_i} exp s_i(a, v).
 *
 * phi_tab, psi_tab : [V, r] vocabulary-wide codebook tables (Eq. ubtree-codebook,
 *            precomputed), dtype feat_dt.  gate : [B, gamma, r] = P(h_i), dtype feat_dt.
 *            r % 16 == 0, 16 <= r <= UBT_MAX_RANK.
 * anchor   : int32 [B] anchor tokens x_0, each in [0, V).
 * cand_ids, cand_logit : outputs of ubt_topk ([B, gamma, K]).
 * alpha, lambda : [host] float [gamma], finite and > 0.
 * delta    : float [B, gamma, K, K] indexed [b][i][a][c] (a = predecessor rank, c =
 *            successor rank); may be NULL.  logq : float [B, gamma, K, K], same
 *            indexing, every entry <= 0.  At i = 0 the predecessor is the anchor: row
 *            a = 0 holds the scores; rows 1..K-1 are written as 0.
 * bf16 features: each product P(h)_k phi_k(a) psi_k(b) is formed exactly in fp32 and
 * summed in fp32 (matrix cores); fp32 features: fp32 fused multiply-adds.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_bigram_scores(const void* phi_tab, const void* psi_tab, const void* gate,
                               ubt_dtype_t feat_dt, int64_t V, int r, const int32_t* anchor,
                               const int32_t* cand_ids, const float* cand_logit,
                               const float* alpha, const float* lambda, int B, int gamma, int K,
                               float* delta, float* logq, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_build_tree -- Algorithm 1 (Appendix A): depth-wise expansion, Eq.
 * (ubtree-frontier), F_d = Top_W(E_d) over all extensions of F_{d-1}; depth bonus, Eq.
 * (ubtree-depth-bonus), l_zeta(y_{1:d}) = l_zeta(y_{1:d-1}) + log q_d^bi + zeta; global
 * pruning, Eq. (ubtree-pruning), T = {root} + Top_budget(union of F_d).
 *
 * Ties: within a depth, score desc, then the parent's position in F_{d-1}, then the
 * candidate rank; across depths, score desc, then depth asc, then that order.  Scores
 * are accumulated in fp32 as (l(parent) + logq) + zeta.
 *
 * anchor, cand_ids : as for ubt_bigram_scores.  logq : [B, gamma, K, K] from
 *            ubt_bigram_scores; entries must be <= 0 (any finite values <= 0 work).
 * W        : search width, 1 <= W <= UBT_MAX_WIDTH, W*K <= UBT_MAX_EXPANSION and
 *            gamma*W <= UBT_MAX_EXPANSION.
 * budget   : non-root node budget (the paper's B), 1 <= budget <= UBT_MAX_BUDGET;
 *            N = budget + 1 tree slots.
 * zeta     : depth bonus, finite and <= 0 (the paper uses 0).
 * n_nodes  : int32 [B] = 1 + min(budget, |union of F_d|).
 * token, parent, depth, cand_rank : int32 [B, N]; score : float [B, N].  Slot 0 is the
 *            root (token = anchor, parent -1, depth 0, cand_rank -1, score 0); slots
 *            1..n_nodes-1 hold the selected nodes in pruning order, which is
 *            topological (parent[n] < n).  Unused slots: -1 and score -inf.
 * mask     : uint32 [B, N, ceil(N/32)] or NULL.  Bit m%32 of word m/32 of row n is set
 *            iff slot m is slot n or an ancestor of it; rows >= n_nodes are zero.
 * dbg      : [host] pointer to a struct of device arrays, or NULL.  When given, receives
 *            the supertree: f_count int32 [B, gamma] = |F_d|; f_parent_slot (the parent's
 *            position in F_{d-1}), f_cand (candidate rank) int32 [B, gamma, W] and
 *            f_score float [B, gamma, W], in F_d order; unused entries -1 / -inf.
 * ------------------------------------------------------------------------------------ */
typedef struct ubt_supertree {
  int32_t* f_count;
  int32_t* f_parent_slot;
  int32_t* f_cand;
  float* f_score;
} ubt_supertree_t;

ubt_status_t ubt_build_tree(const int32_t* anchor, const int32_t* cand_ids, const float* logq,
                            int B, int gamma, int K, int W, int budget, float zeta,
                            int32_t* n_nodes, int32_t* token, int32_t* parent, int32_t* depth,
                            int32_t* cand_rank, float* score, uint32_t* mask,
                            const ubt_supertree_t* dbg, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_draft_tree -- ubt_bigram_scores (without delta) followed by ubt_build_tree
 * (without the supertree) in one call: Method / Parallel Computation, then Algorithm 1.
 * The arguments are those of the two calls, with the same meaning, layout and checks;
 * logq is required and receives the same values.  Every output is bit-identical to
 * that of the two calls.
 *
 * With bf16 features, K in {4, 8, 16}, W <= 64, W*K <= 512 and gamma*W <= 1024, one
 * kernel launch computes each sequence's score slabs in on-chip memory and searches
 * them there (logq is still written out).  Other shapes launch the two calls' kernels
 * in order on `stream`.  In the one-launch kernel the search waits for slabs that other
 * waves of its workgroup compute; each wait is bounded (1 s).  A sequence whose wait ran
 * out of time (a stalled device; never in normal operation) is written with n_nodes = 0
 * and its other outputs are unspecified.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_draft_tree(const void* phi_tab, const void* psi_tab, const void* gate,
                            ubt_dtype_t feat_dt, int64_t V, int r, const int32_t* anchor,
                            const int32_t* cand_ids, const float* cand_logit, const float* alpha,
                            const float* lambda, int B, int gamma, int K, int W, int budget,
                            float zeta, float* logq, int32_t* n_nodes, int32_t* token,
                            int32_t* parent, int32_t* depth, int32_t* cand_rank, float* score,
                            uint32_t* mask, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_draft_step -- one whole draft step: ubt_topk, then ubt_draft_tree, in one call.
 * Method / Unigram Proposer, Eq. (ubtree-unigram) and "Candidate Sets"; Method /
 * Parallel Computation, Eq. (ubtree-edge-matrix); Depth Calibration, Eq.
 * (ubtree-depth); Appendix A / Path Scores, Eq. (ubtree-path); Appendix A, Algorithm 1
 * with Eqs. (ubtree-frontier) and (ubtree-pruning); Verification via Tree-attention.
 *
 * The arguments are those of the two calls with the same meaning, layout and checks
 * (cand_ids, cand_logit and logq are required outputs here).  cand_ids, cand_logit,
 * logq and every tree output are bit-identical to those of ubt_topk followed by
 * ubt_draft_tree; lse and cand_logprob agree to fp32 rounding (the sums run in another
 * order).
 *
 * When the rows are 16-byte aligned, the features are bf16, B <= 64, B is below the
 * device's compute-unit count, and the search shape is one ubt_draft_tree handles in one
 * launch, the step is ONE kernel launch: the rows are swept in depth order, each cut
 * into at most 2 chunks whose LSE and top K are merged per row, while one workgroup per
 * sequence merges each row as soon as its chunks are in, computes the score slab and
 * runs the search.  That launch needs `workspace`: device memory of at least
 * ubt_draft_step_workspace_bytes(B, gamma, V, K, dt) bytes (about
 * 256 + B * gamma * (4 + 2 * (8K + 4))), 256-byte aligned, owned by the caller and
 * ZERO-FILLED before its first use.  It holds an error word (the first 4 bytes), one
 * chunk counter per row (from byte 256) and the chunks' partial results; each call
 * resets the counters it raised, so one workspace serves any number of consecutive calls
 * on one stream; calls that may overlap need separate workspaces.  A chunk's results are
 * exchanged through agent-scope atomic stores and loads, and its row counter is raised
 * only after those stores have completed.  Every wait inside the launch is bounded (1 s).
 * If one runs out of time (a
 * stalled device; never in normal operation) the error word becomes nonzero, the
 * affected sequences are written with n_nodes = 0, the call's outputs are unspecified,
 * and the workspace must be zero-filled again before the next call (a late chunk may
 * still raise a counter).  A missing, short or misaligned workspace returns
 * UBT_ERR_WORKSPACE.
 *
 * With K = 64 (bf16 features, the four-wave search of ubt_draft_tree: W <= 16, B <= 64
 * and below the compute-unit count) the step is TWO launches: the sweep of ubt_topk, then
 * the selector and the search together, one workgroup per sequence searching while the
 * score slabs are computed by other workgroups in depth order; a search waits for each
 * slab (two depths ahead) on a ready word that the slab's workgroup sets once its
 * agent-scope stores have completed.  The ready words are the workspace's row counters
 * (from byte 256, one per row; the same zero-fill, reset, error-word and bounded-wait
 * rules as above).  A missing, short or misaligned workspace here runs the separate
 * kernels instead.  Other shapes run the two calls' kernels in order on `stream` and
 * ignore the workspace.
 * ------------------------------------------------------------------------------------ */
size_t ubt_draft_step_workspace_bytes(int B, int gamma, int64_t V, int K, ubt_dtype_t dt);

ubt_status_t ubt_draft_step(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V,
                            int64_t stride_b, int64_t stride_i, int K, const void* phi_tab,
                            const void* psi_tab, const void* gate, ubt_dtype_t feat_dt, int r,
                            const int32_t* anchor, const float* alpha, const float* lambda, int W,
                            int budget, float zeta, int32_t* cand_ids, float* cand_logit,
                            float* cand_logprob, float* lse, float* logq, int32_t* n_nodes,
                            int32_t* token, int32_t* parent, int32_t* depth, int32_t* cand_rank,
                            float* score, uint32_t* mask, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_draft_step_noalloc -- ubt_draft_step for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments without the workspace, the same checks, kernels and
 * outputs.  It calls no hipMalloc, hipFree or allocating routine.
 *
 * The one-launch kernel's workspace is a static device array of the library
 * (1,097,984 bytes, enough for every shape the one launch takes: B <= 64, gamma <= 64,
 * K <= 16), one per device, held until the process ends; its address is looked up once
 * per device on the first call there.  Each call first clears the error word and the row
 * counters (a small fill kernel on `stream`), so a call never depends on what an earlier
 * one left behind.  Calls that overlap on one device share that array and race: issue
 * them on one stream (or otherwise order them).  A sequence whose bounded wait ran out
 * of time (a stalled device) is written with n_nodes = 0.  A shape whose workspace would
 * exceed the array returns UBT_ERR_WORKSPACE (the one-launch shapes never do); the K = 64
 * selector + search launch keeps its ready words in the same array (cleared the same
 * way); other shapes run the separate kernels, which need no workspace.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_draft_step_noalloc(const void* logits, ubt_dtype_t dt, int B, int gamma,
                                    int64_t V, int64_t stride_b, int64_t stride_i, int K,
                                    const void* phi_tab, const void* psi_tab, const void* gate,
                                    ubt_dtype_t feat_dt, int r, const int32_t* anchor,
                                    const float* alpha, const float* lambda, int W, int budget,
                                    float zeta, int32_t* cand_ids, float* cand_logit,
                                    float* cand_logprob, float* lse, float* logq, int32_t* n_nodes,
                                    int32_t* token, int32_t* parent, int32_t* depth,
                                    int32_t* cand_rank, float* score, uint32_t* mask,
                                    hipStream_t stream);

/* ====================================================================================
 * Unigram-plus-bigram scoring with best-first growth.  Each edge scores its successor's
 * unigram log-probability plus its raw selector score; a path ranks by the cumulative
 * sum, and the tree grows best-first from the root.  Those sums are not monotone along a
 * path (a selector score can exceed the log-probability it is added to), so the prefix
 * closure that Appendix A / Global Pruning gets from normalised scores is enforced by
 * the growth rule instead: a node is eligible only once its parent is in the tree.
 * ==================================================================================== */

/* ------------------------------------------------------------------------------------
 * ubt_edge_scores -- edge scores of the unigram-plus-bigram scoring:
 *   e_i(a, c) = alpha_i log q_i(C_i[c]) + lambda_i delta_i(a, c)
 * with log q_i the unigram log-probability (Method / Unigram Proposer, Eq.
 * ubtree-unigram), delta_i the selector score (Background, Eq. dflash2-selector; Method /
 * Parallel Computation, Eq. ubtree-edge-matrix) and the depth weights of Method / Depth
 * Calibration, Eq. (ubtree-depth); no normalisation over the successors.
 *
 * Arguments as for ubt_bigram_scores, with cand_logprob (ubt_topk's log-probabilities,
 * [B, gamma, K]) in place of cand_logit and `edge` in place of logq: float
 * [B, gamma, K, K] indexed [b][i][a][c], any sign.  At i = 0 row a = 0 (the anchor)
 * holds the scores and rows 1..K-1 are written as 0.  delta may be NULL.  The same
 * matrix-core tile as ubt_bigram_scores forms delta; e = fmaf(lambda, delta, alpha *
 * logprob) in fp32.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_edge_scores(const void* phi_tab, const void* psi_tab, const void* gate,
                             ubt_dtype_t feat_dt, int64_t V, int r, const int32_t* anchor,
                             const int32_t* cand_ids, const float* cand_logprob, const float* alpha,
                             const float* lambda, int B, int gamma, int K, float* delta, float* edge,
                             hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_build_tree_best_first -- best-first growth under cumulative edge scores
 * (Background, "Tree Drafting": best-first search over accumulated scores) with the
 * depth bonus of Appendix A, Eq. (ubtree-depth-bonus):
 *   l(y_{1:d}) = sum_{i<=d} e_i(y_{i-1}, y_i) + zeta * d,  y_0 = the anchor (row 0).
 * From the root (slot 0), `budget` times: among the children of the tree's nodes that
 * are not yet in the tree, the best joins it, under the order score desc, then depth
 * asc, then the parent's slot asc, then candidate rank asc.  Slots follow that growth
 * order, so parent[n] < n; the tree stops early only when the whole lattice is in.
 * Scores accumulate in fp32 as (l(parent) + e) + zeta.
 *
 * anchor, cand_ids : as for ubt_build_tree.  edge : [B, gamma, K, K] from ubt_edge_scores
 *            (any finite values).  K <= UBT_MAX_K, gamma <= UBT_MAX_GAMMA, 1 <= budget <=
 *            UBT_MAX_BUDGET, zeta finite and <= 0.
 * Outputs exactly as ubt_build_tree's (n_nodes, token, parent, depth, cand_rank, score,
 * mask; unused slots -1 / -inf; mask may be NULL), with slots in growth order.
 * One wavefront per sequence; edge slabs of up to 32 KB per sequence are staged in LDS.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_build_tree_best_first(const int32_t* anchor, const int32_t* cand_ids,
                                       const float* edge, int B, int gamma, int K, int budget,
                                       float zeta, int32_t* n_nodes, int32_t* token,
                                       int32_t* parent, int32_t* depth, int32_t* cand_rank,
                                       float* score, uint32_t* mask, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_tree_mask -- the ancestor ("tree attention") mask of a tree given by parent
 * pointers.  Appendix A / Verification via Tree-attention: each node is verified under
 * its own prefix, i.e. it attends to itself and its ancestors.
 *
 * parent   : int32 [B, N] with parent[0] = -1 and 0 <= parent[n] < n for
 *            1 <= n < n_nodes[b]; entries at n >= n_nodes[b] are ignored.
 * n_nodes  : int32 [B], values in [0, N].
 * N        : slots per tree, 1 <= N <= UBT_MAX_BUDGET + 1.
 * mask     : uint32 [B, N, ceil(N/32)], same layout as ubt_build_tree's.  A parent
 *            pointer outside [0, n) ends that row's walk (the row is then unspecified).
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_tree_mask(const int32_t* parent, const int32_t* n_nodes, int B, int N,
                           uint32_t* mask, hipStream_t stream);

/* ====================================================================================
 * Verification of a draft tree (the consumer of the tree and its mask).
 * Appendix A / Verification via Tree-attention; Background, "Tree Drafting".
 * ==================================================================================== */

/* ------------------------------------------------------------------------------------
 * ubt_tree_attention -- attention of every tree node over the committed context and its
 * own ancestors.  Appendix A / Verification via Tree-attention: the whole tree is
 * verified in one target forward pass, each node evaluated under its own
 * autoregressive prefix (the committed tokens, then the root-to-node path).
 *
 * For node n < n_nodes[b] and query head h (key/value head h / (H / H_kv)):
 *   out[b, n, h] = sum_j softmax_j(scale * q[b, n, h] . k_j) v_j
 * over j = the cache positions 0..prefix_len[b]-1 and the tree nodes m < n_nodes[b]
 * whose bit m is set in mask row n (its ancestors and itself, as ubt_build_tree and
 * ubt_tree_mask write it).  lse[b, n, h] = the natural log of the softmax denominator
 * plus its maximum.  Rows n >= n_nodes[b] are written as 0 (lse -inf).
 *
 * q           : bf16 [B, N, H, D], 16-byte aligned.
 * k_cache,
 * v_cache     : bf16 [B, P_max, H_kv, D], 16-byte aligned (may be NULL if P_max == 0).
 * prefix_len  : int32 [B], values clamped to [0, P_max].
 * k_tree,
 * v_tree      : bf16 [B, N, H_kv, D], the keys and values of the tree nodes (root at
 *               slot 0), 16-byte aligned.
 * mask        : uint32 [B, N, ceil(N/32)], LSB-first.
 * n_nodes     : int32 [B], values clamped to [0, N].
 * N           : 1 <= N <= UBT_MAX_BUDGET + 1; H % H_kv == 0; D in {64, 128}
 *               (UBT_ERR_UNSUPPORTED otherwise); scale > 0 and finite.
 * out         : [B, N, H, D] of out_dt (bf16 rounds to nearest even, or f32),
 *               16-byte aligned.
 * lse         : optional float [B, N, H].
 * Products run on bf16 MFMA with fp32 accumulation; the probabilities are rounded to
 * bf16 before the value product.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_tree_attention(const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* prefix_len, int64_t P_max, const void* k_tree,
                                const void* v_tree, const uint32_t* mask, const int32_t* n_nodes,
                                int B, int N, int H, int H_kv, int D, float scale, void* out,
                                ubt_dtype_t out_dt, float* lse, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_verify_accept -- the acceptance walk.  Appendix A / Verification via
 * Tree-attention: from the root, follow the child whose token equals the target model's
 * sample at the current node, until no child matches; that sample is the bonus token.
 *
 * token, parent : int32 [B, N], a tree as ubt_build_tree writes it (parent[n] < n).
 * n_nodes       : int32 [B], clamped to [1, N].
 * target        : int32 [B, N]: target[b, n] is the target's sample after node n's prefix.
 * accept_len    : int32 [B], the number of accepted non-root nodes.
 * accept_nodes  : int32 [B, N]: node 0, then the accepted nodes in path order, then -1.
 * bonus         : int32 [B].
 * Only nodes after the current one are searched, and among several matching children
 * the lowest index is taken, so any input ends the walk within N steps.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_verify_accept(const int32_t* token, const int32_t* parent,
                               const int32_t* n_nodes, const int32_t* target, int B, int N,
                               int32_t* accept_len, int32_t* accept_nodes, int32_t* bonus,
                               hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_commit_kv -- carries the key/value rows of the accepted path into the cache.
 * Appendix A / Verification via Tree-attention: the cache along the accepted path moves
 * on to the next round; other branches are discarded.
 *
 * Copies the rows of nodes accept_nodes[b, 0..accept_len[b]] (the root and the accepted
 * nodes; H_kv * D bf16 each) of k_tree / v_tree [B, N, H_kv, D] to positions
 * prefix_len[b], prefix_len[b] + 1, ... of k_cache / v_cache [B, P_max, H_kv, D], then
 * sets prefix_len[b] += accept_len[b] + 1.  Rows that would land at or past P_max are
 * dropped and prefix_len stops at P_max.  D in {64, 128}; every bf16 array 16-byte
 * aligned.  Calls on one prefix_len array must not overlap.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_commit_kv(const void* k_tree, const void* v_tree, const int32_t* accept_nodes,
                           const int32_t* accept_len, int32_t* prefix_len, void* k_cache,
                           void* v_cache, int B, int N, int H_kv, int D, int64_t P_max,
                           hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * ubt_tree_kl_loss -- UBTree's training objective and its gradients.  Method /
 * Tree-native Training, Eq. (ubtree-training-distributions) and Eq.
 * (ubtree-training-loss).
 *
 * For sequence b and position i (row (b, i), depth i + 1) with ground-truth token
 * y = y_star[b, i] and predecessor a = anchor[b] (i = 0) or y_star[b, i - 1]:
 *   s(c)   = alpha[i] u_i(c) + lambda[i] delta_i(a, c),  delta_i(a, c) = (P(h_i) * phi(a)) . psi(c)
 *   p~(c)  = softmax over c in C_i of z_i(c) / T_train  (T_train = 0: uniform over the
 *            maximisers of z_i on C_i, the limit T -> 0+)
 *   q~(c)  = softmax over c in C_i of s(c)
 *   kl     = sum_c p~ (log p~ - log q~),   ce = -log q_i(y) = lse[b, i] - u_i(y)
 *   loss   = kl + beta * ce
 *   grad_s[b, i, j]      = d loss / d s(C_i[j]) = q~ - p~
 *   grad_logits[b, i, v] = d loss / d u_i(v) = beta (exp(u_i(v) - lse) - [v = y])
 *                          + alpha[i] [v in C_i] (q~ - p~)(v)
 * Positions with y outside [0, V) are not valid: loss, kl, ce, grad_s and the gradient row
 * are 0.  A predecessor outside [0, V) gives delta = 0.
 *
 * logits, dt, B, gamma, V, stride_b, stride_i : the proposer logits u, as for ubt_topk.
 * lse, cand_ids, cand_logit, K : ubt_topk's outputs for these logits (C_i and u_i(C_i));
 *               the ids of one row must be distinct and in [0, V).
 * target_logits : the target logits z, dtype dt, [B, gamma, V] with strides t_stride_b,
 *               t_stride_i (only the entries of C_i are read); finite on C_i.
 * y_star        : int32 [B, gamma]; anchor : int32 [B].
 * phi_tab, psi_tab, gate, feat_dt, r, alpha, lambda : the selector's inputs, with
 *               the checks of ubt_bigram_scores.
 * T_train >= 0, beta >= 0, both finite.
 * loss [B, gamma] required; kl, ce [B, gamma], grad_s [B, gamma, K] and grad_logits
 * float [B, gamma, V] (contiguous, 16-byte aligned) optional.  With grad_logits, two
 * launches: a dense pass over the logits, then the per-position kernel.
 * ------------------------------------------------------------------------------------ */
ubt_status_t ubt_tree_kl_loss(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V,
                              int64_t stride_b, int64_t stride_i, const float* lse,
                              const int32_t* cand_ids, const float* cand_logit, int K,
                              const void* target_logits, int64_t t_stride_b, int64_t t_stride_i,
                              const int32_t* y_star, const int32_t* anchor, const void* phi_tab,
                              const void* psi_tab, const void* gate, ubt_dtype_t feat_dt, int r,
                              const float* alpha, const float* lambda, float T_train, float beta,
                              float* loss, float* kl, float* ce, float* grad_s, float* grad_logits,
                              hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* UBT_H */
