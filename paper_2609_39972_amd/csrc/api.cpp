// Host side of libubt.so: argument validation and kernel launches for the C ABI
// declared in include/ubt.h.  Every check runs before any launch; on an error status
// nothing is launched.
#include <math.h>
#include <stdint.h>

#include "ubt.h"
#include "ubt_launch.h"

namespace {

thread_local int g_last_hip_error = 0;

ubt_status_t hip_status(hipError_t e) {
  if (e == hipSuccess) return UBT_OK;
  g_last_hip_error = static_cast<int>(e);
  return UBT_ERR_HIP;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_dtype(ubt_dtype_t dt) { return dt == UBT_F32 || dt == UBT_BF16; }

// Checks of ubt_bigram_scores' arguments (logq and delta aside); fills the scales.
ubt_status_t check_selector(const void* phi_tab, const void* psi_tab, const void* gate, ubt_dtype_t feat_dt, int64_t V,
                            int r, const int32_t* anchor, const int32_t* cand_ids, const float* cand_logit,
                            const float* alpha, const float* lambda, int B, int gamma, int K, ubt::Scales& sc) {
  if (!phi_tab || !psi_tab || !gate || !anchor || !cand_ids || !cand_logit || !alpha || !lambda) return UBT_ERR_NULL;
  if (!valid_dtype(feat_dt)) return UBT_ERR_VALUE;
  if (B < 1 || gamma < 1 || gamma > UBT_MAX_GAMMA || K < 1 || K > UBT_MAX_K || V < K || V >= (int64_t(1) << 31))
    return UBT_ERR_SHAPE;
  if (r < 16 || r > UBT_MAX_RANK || r % 16 != 0) return UBT_ERR_SHAPE;
  for (int i = 0; i < gamma; ++i)
    if (!(isfinite(alpha[i]) && alpha[i] > 0.f && isfinite(lambda[i]) && lambda[i] > 0.f)) return UBT_ERR_VALUE;
  if (feat_dt == UBT_BF16 && !(aligned16(phi_tab) && aligned16(psi_tab) && aligned16(gate)))
    return UBT_ERR_UNSUPPORTED;
  sc = ubt::Scales{};
  for (int i = 0; i < gamma; ++i) {
    sc.alpha[i] = alpha[i];
    sc.lambda[i] = lambda[i];
  }
  return UBT_OK;
}

// Checks of ubt_build_tree's arguments (logq and dbg aside); fills the launch arguments.
ubt_status_t check_tree(const int32_t* anchor, const int32_t* cand_ids, int B, int gamma, int K, int W, int budget,
                        float zeta, int32_t* n_nodes, int32_t* token, int32_t* parent, int32_t* depth,
                        int32_t* cand_rank, float* score, uint32_t* mask, ubt::TreeArgs& a) {
  if (!anchor || !cand_ids || !n_nodes || !token || !parent || !depth || !cand_rank || !score) return UBT_ERR_NULL;
  if (B < 1 || gamma < 1 || gamma > UBT_MAX_GAMMA || K < 1 || K > UBT_MAX_K) return UBT_ERR_SHAPE;
  if (W < 1 || W > UBT_MAX_WIDTH || budget < 1 || budget > UBT_MAX_BUDGET) return UBT_ERR_SHAPE;
  if (static_cast<int64_t>(W) * K > UBT_MAX_EXPANSION || static_cast<int64_t>(gamma) * W > UBT_MAX_EXPANSION)
    return UBT_ERR_UNSUPPORTED;
  if (!(isfinite(zeta) && zeta <= 0.f)) return UBT_ERR_VALUE;
  a = ubt::TreeArgs{};
  a.anchor = anchor;
  a.cand_ids = cand_ids;
  a.B = B;
  a.gamma = gamma;
  a.K = K;
  a.W = W;
  a.budget = budget;
  a.zeta = zeta;
  a.n_nodes = n_nodes;
  a.token = token;
  a.parent = parent;
  a.depth = depth;
  a.cand_rank = cand_rank;
  a.score = score;
  a.mask = mask;
  return UBT_OK;
}

}  // namespace

extern "C" {

const char* ubt_status_str(ubt_status_t s) {
  switch (s) {
    case UBT_OK: return "UBT_OK";
    case UBT_ERR_NULL: return "UBT_ERR_NULL";
    case UBT_ERR_SHAPE: return "UBT_ERR_SHAPE";
    case UBT_ERR_VALUE: return "UBT_ERR_VALUE";
    case UBT_ERR_UNSUPPORTED: return "UBT_ERR_UNSUPPORTED";
    case UBT_ERR_WORKSPACE: return "UBT_ERR_WORKSPACE";
    case UBT_ERR_HIP: return "UBT_ERR_HIP";
  }
  return "UBT_ERR_UNKNOWN";
}

int ubt_abi_version(void) { return UBT_ABI_VERSION; }

int ubt_last_hip_error(void) { return g_last_hip_error; }

ubt_status_t ubt_topk(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V, int64_t stride_b,
                      int64_t stride_i, int K, int32_t* cand_ids, float* cand_logit, float* cand_logprob, float* lse,
                      hipStream_t stream) {
  if (!logits || !cand_ids || !cand_logit) return UBT_ERR_NULL;
  if (!valid_dtype(dt)) return UBT_ERR_VALUE;
  if (B < 1 || gamma < 1 || gamma > UBT_MAX_GAMMA || K < 1 || K > UBT_MAX_K || V < K || V >= (int64_t(1) << 31))
    return UBT_ERR_SHAPE;
  if (stride_i < V || stride_b < static_cast<int64_t>(gamma) * stride_i) return UBT_ERR_SHAPE;
  if (static_cast<int64_t>(B) * gamma > 0x7FFFFFFF) return UBT_ERR_SHAPE;
  if (V * (dt == UBT_BF16 ? 2 : 4) >= (int64_t(1) << 32)) return UBT_ERR_SHAPE;  // a row is one buffer range
  const int64_t es = dt == UBT_BF16 ? 2 : 4;
  const bool aligned = aligned16(logits) && (stride_b * es) % 16 == 0 && (stride_i * es) % 16 == 0;
  return hip_status(ubt::launch_topk(logits, static_cast<int>(dt), aligned, B, gamma, V, stride_b, stride_i, K,
                                     cand_ids, cand_logit, cand_logprob, lse, stream));
}

size_t ubt_lm_head_topk_workspace_bytes(int M, int d, int64_t V, int K) {
  if (M < 1 || d < 32 || d > 65536 || d % 32 != 0 || K < 1 || K > UBT_MAX_K || V < K || V >= (int64_t(1) << 31))
    return 0;
  return ubt::lm_head_workspace_bytes(M, d, V, K);
}

ubt_status_t ubt_lm_head_topk(const void* h, const void* w_lm, int M, int d, int64_t V, int K, int32_t* cand_ids,
                              float* cand_logit, float* cand_logprob, float* lse, void* workspace, size_t ws_bytes,
                              hipStream_t stream) {
  if (!h || !w_lm || !cand_ids || !cand_logit) return UBT_ERR_NULL;
  if (M < 1 || d < 32 || d > 65536 || d % 32 != 0 || K < 1 || K > UBT_MAX_K || V < K || V >= (int64_t(1) << 31))
    return UBT_ERR_SHAPE;
  if (!aligned16(h) || !aligned16(w_lm)) return UBT_ERR_UNSUPPORTED;
  const size_t need = ubt::lm_head_workspace_bytes(M, d, V, K);
  if (need == 0) return UBT_ERR_UNSUPPORTED;
  if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return UBT_ERR_WORKSPACE;
  return hip_status(ubt::launch_lm_head_topk(h, w_lm, M, d, V, K, cand_ids, cand_logit, cand_logprob, lse, workspace,
                                             stream));
}

ubt_status_t ubt_bigram_scores(const void* phi_tab, const void* psi_tab, const void* gate, ubt_dtype_t feat_dt,
                               int64_t V, int r, const int32_t* anchor, const int32_t* cand_ids,
                               const float* cand_logit, const float* alpha, const float* lambda, int B, int gamma,
                               int K, float* delta, float* logq, hipStream_t stream) {
  if (!logq) return UBT_ERR_NULL;
  ubt::Scales sc;
  const ubt_status_t st = check_selector(phi_tab, psi_tab, gate, feat_dt, V, r, anchor, cand_ids, cand_logit, alpha,
                                         lambda, B, gamma, K, sc);
  if (st != UBT_OK) return st;
  return hip_status(ubt::launch_bigram(phi_tab, psi_tab, gate, static_cast<int>(feat_dt), V, r, anchor, cand_ids,
                                       cand_logit, sc, B, gamma, K, delta, logq, stream));
}

ubt_status_t ubt_build_tree(const int32_t* anchor, const int32_t* cand_ids, const float* logq, int B, int gamma, int K,
                            int W, int budget, float zeta, int32_t* n_nodes, int32_t* token, int32_t* parent,
                            int32_t* depth, int32_t* cand_rank, float* score, uint32_t* mask,
                            const ubt_supertree_t* dbg, hipStream_t stream) {
  if (!logq) return UBT_ERR_NULL;
  if (dbg && !(dbg->f_count && dbg->f_parent_slot && dbg->f_cand && dbg->f_score)) return UBT_ERR_NULL;
  ubt::TreeArgs a;
  const ubt_status_t st = check_tree(anchor, cand_ids, B, gamma, K, W, budget, zeta, n_nodes, token, parent, depth,
                                     cand_rank, score, mask, a);
  if (st != UBT_OK) return st;
  a.logq = logq;
  if (dbg) {
    a.f_count = dbg->f_count;
    a.f_parent = dbg->f_parent_slot;
    a.f_cand = dbg->f_cand;
    a.f_score = dbg->f_score;
  }
  return hip_status(ubt::launch_build_tree(a, stream));
}

ubt_status_t ubt_draft_tree(const void* phi_tab, const void* psi_tab, const void* gate, ubt_dtype_t feat_dt,
                            int64_t V, int r, const int32_t* anchor, const int32_t* cand_ids, const float* cand_logit,
                            const float* alpha, const float* lambda, int B, int gamma, int K, int W, int budget,
                            float zeta, float* logq, int32_t* n_nodes, int32_t* token, int32_t* parent,
                            int32_t* depth, int32_t* cand_rank, float* score, uint32_t* mask, hipStream_t stream) {
  if (!logq) return UBT_ERR_NULL;
  ubt::Scales sc;
  ubt_status_t st = check_selector(phi_tab, psi_tab, gate, feat_dt, V, r, anchor, cand_ids, cand_logit, alpha, lambda,
                                   B, gamma, K, sc);
  if (st != UBT_OK) return st;
  ubt::TreeArgs a;
  st = check_tree(anchor, cand_ids, B, gamma, K, W, budget, zeta, n_nodes, token, parent, depth, cand_rank, score,
                  mask, a);
  if (st != UBT_OK) return st;
  a.logq = logq;
  if (ubt::draft_tree_fused(static_cast<int>(feat_dt), gamma, K, W)) {
    ubt::SelectorArgs s;
    s.phi = static_cast<const uint16_t*>(phi_tab);
    s.psi = static_cast<const uint16_t*>(psi_tab);
    s.gate = static_cast<const uint16_t*>(gate);
    s.V = V;
    s.r = r;
    s.cand_logit = cand_logit;
    s.logq = logq;
    s.sc = sc;
    return hip_status(ubt::launch_draft_tree(s, a, stream));
  }
  st = hip_status(ubt::launch_bigram(phi_tab, psi_tab, gate, static_cast<int>(feat_dt), V, r, anchor, cand_ids,
                                     cand_logit, sc, B, gamma, K, nullptr, logq, stream));
  if (st != UBT_OK) return st;
  return hip_status(ubt::launch_build_tree(a, stream));
}

size_t ubt_draft_step_workspace_bytes(int B, int gamma, int64_t V, int K, ubt_dtype_t dt) {
  if (B < 1 || gamma < 1 || gamma > UBT_MAX_GAMMA || K < 1 || K > UBT_MAX_K || V < K || V >= (int64_t(1) << 31) ||
      !valid_dtype(dt))
    return 0;
  return ubt::step_workspace_bytes(B, gamma, V, K, dt == UBT_BF16 ? 1 : 0);
}

}  // extern "C"

namespace {

// ubt_draft_step and ubt_draft_step_noalloc: the same checks and kernels; the one-launch
// kernel's workspace is the caller's (use_static = false) or the library's static array.
ubt_status_t draft_step_impl(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V, int64_t stride_b,
                             int64_t stride_i, int K, const void* phi_tab, const void* psi_tab, const void* gate,
                             ubt_dtype_t feat_dt, int r, const int32_t* anchor, const float* alpha,
                             const float* lambda, int W, int budget, float zeta, int32_t* cand_ids, float* cand_logit,
                             float* cand_logprob, float* lse, float* logq, int32_t* n_nodes, int32_t* token,
                             int32_t* parent, int32_t* depth, int32_t* cand_rank, float* score, uint32_t* mask,
                             void* workspace, size_t workspace_bytes, bool use_static, hipStream_t stream) {
  if (!logits || !cand_ids || !cand_logit || !logq) return UBT_ERR_NULL;
  if (!valid_dtype(dt)) return UBT_ERR_VALUE;
  if (B < 1 || gamma < 1 || gamma > UBT_MAX_GAMMA || K < 1 || K > UBT_MAX_K || V < K || V >= (int64_t(1) << 31))
    return UBT_ERR_SHAPE;
  if (stride_i < V || stride_b < static_cast<int64_t>(gamma) * stride_i) return UBT_ERR_SHAPE;
  if (V * (dt == UBT_BF16 ? 2 : 4) >= (int64_t(1) << 32)) return UBT_ERR_SHAPE;
  ubt::Scales sc;
  ubt_status_t st = check_selector(phi_tab, psi_tab, gate, feat_dt, V, r, anchor, cand_ids, cand_logit, alpha, lambda,
                                   B, gamma, K, sc);
  if (st != UBT_OK) return st;
  ubt::TreeArgs a;
  st = check_tree(anchor, cand_ids, B, gamma, K, W, budget, zeta, n_nodes, token, parent, depth, cand_rank, score,
                  mask, a);
  if (st != UBT_OK) return st;
  a.logq = logq;
  const int64_t es = dt == UBT_BF16 ? 2 : 4;
  const bool aligned = aligned16(logits) && (stride_b * es) % 16 == 0 && (stride_i * es) % 16 == 0;
  ubt::SelectorArgs s;
  s.phi = static_cast<const uint16_t*>(phi_tab);
  s.psi = static_cast<const uint16_t*>(psi_tab);
  s.gate = static_cast<const uint16_t*>(gate);
  s.V = V;
  s.r = r;
  s.cand_logit = cand_logit;
  s.logq = logq;
  s.sc = sc;
  if (!ubt::draft_step_fused(static_cast<int>(dt), aligned, B, gamma, V, K, static_cast<int>(feat_dt), W)) {
    st = hip_status(ubt::launch_topk(logits, static_cast<int>(dt), aligned, B, gamma, V, stride_b, stride_i, K,
                                     cand_ids, cand_logit, cand_logprob, lse, stream));
    if (st != UBT_OK) return st;
    // K = 64: the selector and the search in one launch when a workspace is at hand.
    if (ubt::draft_step_k64(static_cast<int>(feat_dt), B, gamma, K, W)) {
      const size_t need = ubt::step_k64_workspace_bytes(B, gamma);
      if (use_static && need <= ubt::step_static_scratch_bytes()) {
        st = hip_status(ubt::step_static_scratch(&workspace));
        if (st != UBT_OK) return st;
        st = hip_status(ubt::clear_step_flags(workspace, B, gamma, stream));
        if (st != UBT_OK) return st;
        return hip_status(ubt::launch_draft_step_k64(s, a, workspace, stream));
      }
      if (!use_static && workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u) == 0 && workspace_bytes >= need)
        return hip_status(ubt::launch_draft_step_k64(s, a, workspace, stream));
    }
    return ubt_draft_tree(phi_tab, psi_tab, gate, feat_dt, V, r, anchor, cand_ids, cand_logit, alpha, lambda, B,
                          gamma, K, W, budget, zeta, logq, n_nodes, token, parent, depth, cand_rank, score, mask,
                          stream);
  }
  const size_t need = ubt::step_workspace_bytes(B, gamma, V, K, static_cast<int>(dt));
  if (use_static) {
    if (need > ubt::step_static_scratch_bytes()) return UBT_ERR_WORKSPACE;
    st = hip_status(ubt::step_static_scratch(&workspace));
    if (st != UBT_OK) return st;
    // Every call starts from a clear error word and clear row counters, whatever an
    // earlier call on this device left behind.
    st = hip_status(ubt::clear_step_flags(workspace, B, gamma, stream));
    if (st != UBT_OK) return st;
  } else if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0 || workspace_bytes < need) {
    return UBT_ERR_WORKSPACE;
  }
  return hip_status(ubt::launch_draft_step(logits, static_cast<int>(dt), B, gamma, V, stride_b, stride_i, K, cand_ids,
                                           cand_logit, cand_logprob, lse, s, a, workspace, stream));
}

}  // namespace

extern "C" {

ubt_status_t ubt_draft_step(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V, int64_t stride_b,
                            int64_t stride_i, int K, const void* phi_tab, const void* psi_tab, const void* gate,
                            ubt_dtype_t feat_dt, int r, const int32_t* anchor, const float* alpha,
                            const float* lambda, int W, int budget, float zeta, int32_t* cand_ids, float* cand_logit,
                            float* cand_logprob, float* lse, float* logq, int32_t* n_nodes, int32_t* token,
                            int32_t* parent, int32_t* depth, int32_t* cand_rank, float* score, uint32_t* mask,
                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return draft_step_impl(logits, dt, B, gamma, V, stride_b, stride_i, K, phi_tab, psi_tab, gate, feat_dt, r, anchor,
                         alpha, lambda, W, budget, zeta, cand_ids, cand_logit, cand_logprob, lse, logq, n_nodes,
                         token, parent, depth, cand_rank, score, mask, workspace, workspace_bytes, false, stream);
}

ubt_status_t ubt_draft_step_noalloc(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V,
                                    int64_t stride_b, int64_t stride_i, int K, const void* phi_tab,
                                    const void* psi_tab, const void* gate, ubt_dtype_t feat_dt, int r,
                                    const int32_t* anchor, const float* alpha, const float* lambda, int W,
                                    int budget, float zeta, int32_t* cand_ids, float* cand_logit,
                                    float* cand_logprob, float* lse, float* logq, int32_t* n_nodes, int32_t* token,
                                    int32_t* parent, int32_t* depth, int32_t* cand_rank, float* score,
                                    uint32_t* mask, hipStream_t stream) {
  return draft_step_impl(logits, dt, B, gamma, V, stride_b, stride_i, K, phi_tab, psi_tab, gate, feat_dt, r, anchor,
                         alpha, lambda, W, budget, zeta, cand_ids, cand_logit, cand_logprob, lse, logq, n_nodes,
                         token, parent, depth, cand_rank, score, mask, nullptr, 0, true, stream);
}

ubt_status_t ubt_edge_scores(const void* phi_tab, const void* psi_tab, const void* gate, ubt_dtype_t feat_dt,
                             int64_t V, int r, const int32_t* anchor, const int32_t* cand_ids,
                             const float* cand_logprob, const float* alpha, const float* lambda, int B, int gamma,
                             int K, float* delta, float* edge, hipStream_t stream) {
  if (!edge) return UBT_ERR_NULL;
  ubt::Scales sc;
  const ubt_status_t st = check_selector(phi_tab, psi_tab, gate, feat_dt, V, r, anchor, cand_ids, cand_logprob, alpha,
                                         lambda, B, gamma, K, sc);
  if (st != UBT_OK) return st;
  return hip_status(ubt::launch_bigram(phi_tab, psi_tab, gate, static_cast<int>(feat_dt), V, r, anchor, cand_ids,
                                       cand_logprob, sc, B, gamma, K, delta, edge, stream, false));
}

ubt_status_t ubt_build_tree_best_first(const int32_t* anchor, const int32_t* cand_ids, const float* edge, int B,
                                       int gamma, int K, int budget, float zeta, int32_t* n_nodes, int32_t* token,
                                       int32_t* parent, int32_t* depth, int32_t* cand_rank, float* score,
                                       uint32_t* mask, hipStream_t stream) {
  if (!edge) return UBT_ERR_NULL;
  ubt::TreeArgs a;
  // W does not apply to best-first growth; 1 passes the shared checks.
  const ubt_status_t st = check_tree(anchor, cand_ids, B, gamma, K, 1, budget, zeta, n_nodes, token, parent, depth,
                                     cand_rank, score, mask, a);
  if (st != UBT_OK) return st;
  a.logq = edge;
  return hip_status(ubt::launch_best_first(a, stream));
}

ubt_status_t ubt_tree_mask(const int32_t* parent, const int32_t* n_nodes, int B, int N, uint32_t* mask,
                           hipStream_t stream) {
  if (!parent || !n_nodes || !mask) return UBT_ERR_NULL;
  if (B < 1 || N < 1 || N > UBT_MAX_BUDGET + 1) return UBT_ERR_SHAPE;
  return hip_status(ubt::launch_tree_mask(parent, n_nodes, B, N, mask, stream));
}

ubt_status_t ubt_tree_attention(const void* q, const void* k_cache, const void* v_cache, const int32_t* prefix_len,
                                int64_t P_max, const void* k_tree, const void* v_tree, const uint32_t* mask,
                                const int32_t* n_nodes, int B, int N, int H, int H_kv, int D, float scale, void* out,
                                ubt_dtype_t out_dt, float* lse, hipStream_t stream) {
  if (!q || !prefix_len || !k_tree || !v_tree || !mask || !n_nodes || !out) return UBT_ERR_NULL;
  if (P_max > 0 && (!k_cache || !v_cache)) return UBT_ERR_NULL;
  if (B < 1 || N < 1 || N > UBT_MAX_BUDGET + 1 || H < 1 || H_kv < 1 || H % H_kv != 0 || P_max < 0 ||
      P_max >= (int64_t(1) << 31))
    return UBT_ERR_SHAPE;
  if (D != 64 && D != 128) return UBT_ERR_UNSUPPORTED;
  if (!valid_dtype(out_dt)) return UBT_ERR_VALUE;
  if (!(isfinite(scale) && scale > 0.f)) return UBT_ERR_VALUE;
  const int64_t rows = static_cast<int64_t>(N) * (H / H_kv);
  if (static_cast<int64_t>(B) * H_kv * ((rows + 63) / 64) >= (int64_t(1) << 31)) return UBT_ERR_SHAPE;
  if (!aligned16(q) || !aligned16(k_tree) || !aligned16(v_tree) || !aligned16(out) ||
      (P_max > 0 && (!aligned16(k_cache) || !aligned16(v_cache))))
    return UBT_ERR_UNSUPPORTED;
  ubt::TreeAttnArgs a{};
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.prefix_len = prefix_len;
  a.k_tree = k_tree;
  a.v_tree = v_tree;
  a.mask = mask;
  a.n_nodes = n_nodes;
  a.B = B;
  a.N = N;
  a.H = H;
  a.Hkv = H_kv;
  a.D = D;
  a.Pmax = P_max;
  a.scale = scale;
  a.out = out;
  a.out_f32 = out_dt == UBT_F32 ? 1 : 0;
  a.lse = lse;
  return hip_status(ubt::launch_tree_attention(a, stream));
}

ubt_status_t ubt_verify_accept(const int32_t* token, const int32_t* parent, const int32_t* n_nodes,
                               const int32_t* target, int B, int N, int32_t* accept_len, int32_t* accept_nodes,
                               int32_t* bonus, hipStream_t stream) {
  if (!token || !parent || !n_nodes || !target || !accept_len || !accept_nodes || !bonus) return UBT_ERR_NULL;
  if (B < 1 || N < 1 || N > UBT_MAX_BUDGET + 1) return UBT_ERR_SHAPE;
  return hip_status(
      ubt::launch_verify_accept(token, parent, n_nodes, target, B, N, accept_len, accept_nodes, bonus, stream));
}

ubt_status_t ubt_commit_kv(const void* k_tree, const void* v_tree, const int32_t* accept_nodes,
                           const int32_t* accept_len, int32_t* prefix_len, void* k_cache, void* v_cache, int B, int N,
                           int H_kv, int D, int64_t P_max, hipStream_t stream) {
  if (!k_tree || !v_tree || !accept_nodes || !accept_len || !prefix_len || !k_cache || !v_cache) return UBT_ERR_NULL;
  if (B < 1 || N < 1 || N > UBT_MAX_BUDGET + 1 || H_kv < 1 || P_max < 1 || P_max >= (int64_t(1) << 31))
    return UBT_ERR_SHAPE;
  if (D != 64 && D != 128) return UBT_ERR_UNSUPPORTED;
  if (!aligned16(k_tree) || !aligned16(v_tree) || !aligned16(k_cache) || !aligned16(v_cache))
    return UBT_ERR_UNSUPPORTED;
  return hip_status(ubt::launch_commit_kv(k_tree, v_tree, accept_nodes, accept_len, prefix_len, k_cache, v_cache, B,
                                          N, H_kv, D, P_max, stream));
}

ubt_status_t ubt_tree_kl_loss(const void* logits, ubt_dtype_t dt, int B, int gamma, int64_t V, int64_t stride_b,
                              int64_t stride_i, const float* lse, const int32_t* cand_ids, const float* cand_logit,
                              int K, const void* target_logits, int64_t t_stride_b, int64_t t_stride_i,
                              const int32_t* y_star, const int32_t* anchor, const void* phi_tab, const void* psi_tab,
                              const void* gate, ubt_dtype_t feat_dt, int r, const float* alpha, const float* lambda,
                              float T_train, float beta, float* loss, float* kl, float* ce, float* grad_s,
                              float* grad_logits, hipStream_t stream) {
  if (!logits || !lse || !target_logits || !y_star || !loss) return UBT_ERR_NULL;
  if (!valid_dtype(dt)) return UBT_ERR_VALUE;
  ubt::Scales sc;
  ubt_status_t st = check_selector(phi_tab, psi_tab, gate, feat_dt, V, r, anchor, cand_ids, cand_logit, alpha, lambda,
                                   B, gamma, K, sc);
  if (st != UBT_OK) return st;
  if (stride_i < V || stride_b < static_cast<int64_t>(gamma) * stride_i || t_stride_i < V ||
      t_stride_b < static_cast<int64_t>(gamma) * t_stride_i)
    return UBT_ERR_SHAPE;
  if (static_cast<int64_t>(B) * gamma >= (int64_t(1) << 31) || (V + 8191) / 8192 > 65535) return UBT_ERR_SHAPE;
  if (!(isfinite(T_train) && T_train >= 0.f && isfinite(beta) && beta >= 0.f)) return UBT_ERR_VALUE;
  if (feat_dt == UBT_F32 && !(aligned16(phi_tab) && aligned16(psi_tab) && aligned16(gate))) return UBT_ERR_UNSUPPORTED;
  if (grad_logits && !aligned16(grad_logits)) return UBT_ERR_UNSUPPORTED;
  const int64_t es = dt == UBT_BF16 ? 2 : 4;
  ubt::TreeKlArgs a{};
  a.logits = logits;
  a.target = target_logits;
  a.dtype = static_cast<int>(dt);
  a.feat_dtype = static_cast<int>(feat_dt);
  a.B = B;
  a.gamma = gamma;
  a.K = K;
  a.r = r;
  a.V = V;
  a.stride_b = stride_b;
  a.stride_i = stride_i;
  a.t_stride_b = t_stride_b;
  a.t_stride_i = t_stride_i;
  a.vec = V % 8 == 0 && aligned16(logits) && (stride_b * es) % 16 == 0 && (stride_i * es) % 16 == 0;
  a.lse = lse;
  a.cand_ids = cand_ids;
  a.cand_logit = cand_logit;
  a.y_star = y_star;
  a.anchor = anchor;
  a.phi = phi_tab;
  a.psi = psi_tab;
  a.gate = gate;
  a.sc = sc;
  a.T = T_train;
  a.beta = beta;
  a.loss = loss;
  a.kl = kl;
  a.ce = ce;
  a.grad_s = grad_s;
  a.grad = grad_logits;
  return hip_status(ubt::launch_tree_kl_loss(a, stream));
}

}  // extern "C"
