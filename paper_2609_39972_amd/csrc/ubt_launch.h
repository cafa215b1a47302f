// Internal launch interface between the host API (api.cpp) and the HIP kernels.
// Arguments have been validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ubt {

// ---- top-K sweep --------------------------------------------------------------------
hipError_t launch_topk(const void* logits, int dtype, bool aligned, int B, int gamma, int64_t V,
                       int64_t stride_b, int64_t stride_i, int K, int32_t* cand_ids, float* cand_logit,
                       float* cand_logprob, float* lse, hipStream_t stream);

// ---- selector scores ------------------------------------------------------------------
struct Scales {
  float alpha[64];
  float lambda[64];
};
size_t lm_head_workspace_bytes(int M, int d, int64_t V, int K);
hipError_t launch_lm_head_topk(const void* h, const void* w_lm, int M, int d, int64_t V, int K, int32_t* cand_ids,
                               float* cand_logit, float* cand_logprob, float* lse, void* workspace,
                               hipStream_t stream);
hipError_t launch_bigram(const void* phi, const void* psi, const void* gate, int feat_dtype, int64_t V, int r,
                         const int32_t* anchor, const int32_t* cand_ids, const float* cand_logit,
                         const Scales& scales, int B, int gamma, int K, float* delta, float* logq,
                         hipStream_t stream, bool normalise = true);

// ---- tree search --------------------------------------------------------------------
struct TreeArgs {
  const int32_t* anchor;
  const int32_t* cand_ids;
  const float* logq;
  int B, gamma, K, W, budget;
  float zeta;
  int32_t* n_nodes;
  int32_t* token;
  int32_t* parent;
  int32_t* depth;
  int32_t* cand_rank;
  float* score;
  uint32_t* mask;
  int32_t* f_count;
  int32_t* f_parent;
  int32_t* f_cand;
  float* f_score;
  uint32_t* err;  // one-launch kernels: error word set when a wait inside the launch timed out (may be null)
};
hipError_t launch_build_tree(const TreeArgs& a, hipStream_t stream);

// Best-first tree under cumulative edge scores (edge [B, gamma, K, K]); the tree outputs
// of TreeArgs (logq = the edge scores; W and the supertree unused).
hipError_t launch_best_first(const TreeArgs& a, hipStream_t stream);

hipError_t launch_tree_mask(const int32_t* parent, const int32_t* n_nodes, int B, int N, uint32_t* mask,
                            hipStream_t stream);

// ---- selector scores + tree search in one launch --------------------------------------
struct SelectorArgs {
  const uint16_t* phi;  // bf16 tables and gate
  const uint16_t* psi;
  const uint16_t* gate;
  int64_t V;
  int r;
  const float* cand_logit;
  float* logq;  // also written, [B, gamma, K, K]
  Scales sc;
};
// True if the one-launch kernel handles the shape (bf16 features and the register-
// resident search: K in {4, 8, 16}, W <= 64, W*K <= 512, gamma*W <= 1024).
bool draft_tree_fused(int feat_dtype, int gamma, int K, int W);
// True if draft_tree_k64_kernel handles the shape (bf16 features, K = 64 and the
// four-wave search: W*64 <= 1024, W <= 64, gamma*W <= 1024).
bool draft_tree_k64_fused(int feat_dtype, int gamma, int K, int W);
// Selector scores and the K = 64 search in one launch; ready: B*gamma zero words, left zero.
hipError_t launch_draft_tree_k64(const SelectorArgs& s, const TreeArgs& a, uint32_t* ready, hipStream_t stream);
hipError_t launch_draft_tree(const SelectorArgs& s, const TreeArgs& a, hipStream_t stream);

// ---- the whole step: depth-major chunked sweep beside per-sequence searchers ----------
constexpr int kMaxStepSequences = 64;   // searcher workgroups
// Workspace bytes of launch_draft_step: an error word, one chunk counter per row and the
// chunks' partial results (dtype 1 = bf16 logits, 0 = fp32).
size_t step_workspace_bytes(int B, int gamma, int64_t V, int K, int dtype);
// True if the one-launch step handles the shape: aligned rows, bf16 features, the
// register-resident search, B <= kMaxStepSequences, and fewer sequences than compute
// units (the searchers and the workers are resident together).
bool draft_step_fused(int dtype, bool aligned, int B, int gamma, int64_t V, int K, int feat_dtype, int W);
hipError_t launch_draft_step(const void* logits, int dtype, int B, int gamma, int64_t V, int64_t stride_b,
                             int64_t stride_i, int K, int32_t* cand_ids, float* cand_logit, float* cand_logprob,
                             float* lse, const SelectorArgs& s, const TreeArgs& a, void* workspace,
                             hipStream_t stream);
// The allocation-free variant's workspace: a static device array of
// step_static_scratch_bytes() bytes per device; *ptr receives its address on the current
// device (looked up once per device).
size_t step_static_scratch_bytes();
hipError_t step_static_scratch(void** ptr);
// Zero-fills the error word and the B * gamma row counters of a step workspace.
hipError_t clear_step_flags(void* workspace, int B, int gamma, hipStream_t stream);
// K = 64: the step is the sweep, then draft_tree_k64_kernel, whose slab ready words are
// the workspace's row counters (the error word first, the words from byte 256).  True if
// that launch takes the shape: bf16 features, K = 64, the four-wave search, B <=
// kMaxStepSequences and fewer sequences than compute units (the searchers and the slab
// workgroups are resident together).
bool draft_step_k64(int feat_dtype, int B, int gamma, int K, int W);
size_t step_k64_workspace_bytes(int B, int gamma);
hipError_t launch_draft_step_k64(const SelectorArgs& s, const TreeArgs& a, void* workspace, hipStream_t stream);

// ---- verification: tree attention, acceptance walk, KV commit -------------------------
struct TreeAttnArgs {
  const void* q;        // bf16 [B, N, H, D]
  const void* k_cache;  // bf16 [B, Pmax, Hkv, D]
  const void* v_cache;
  const int32_t* prefix_len;  // [B]
  const void* k_tree;   // bf16 [B, N, Hkv, D]
  const void* v_tree;
  const uint32_t* mask;  // [B, N, ceil(N / 32)]
  const int32_t* n_nodes;
  int B, N, H, Hkv, D;
  int64_t Pmax;
  float scale;
  void* out;  // [B, N, H, D], bf16 or f32
  int out_f32;
  float* lse;  // optional [B, N, H]
};
hipError_t launch_tree_attention(const TreeAttnArgs& a, hipStream_t stream);
hipError_t launch_verify_accept(const int32_t* token, const int32_t* parent, const int32_t* n_nodes,
                                const int32_t* target, int B, int N, int32_t* accept_len, int32_t* accept_nodes,
                                int32_t* bonus, hipStream_t stream);
hipError_t launch_commit_kv(const void* k_tree, const void* v_tree, const int32_t* accept_nodes,
                            const int32_t* accept_len, int32_t* prefix_len, void* k_cache, void* v_cache, int B, int N,
                            int Hkv, int D, int64_t Pmax, hipStream_t stream);

// ---- renormalised-KL training objective -------------------------------------------------
struct TreeKlArgs {
  const void* logits;  // [B, gamma, V] with strides, dtype
  const void* target;  // same dtype, its own strides
  int dtype, feat_dtype, B, gamma, K, r;
  int64_t V, stride_b, stride_i, t_stride_b, t_stride_i;
  bool vec;  // 16-byte aligned rows of V % 8 == 0 elements
  const float* lse;
  const int32_t* cand_ids;
  const float* cand_logit;
  const int32_t* y_star;
  const int32_t* anchor;
  const void* phi;
  const void* psi;
  const void* gate;
  Scales sc;
  float T, beta;
  float* loss;
  float* kl;
  float* ce;
  float* grad_s;
  float* grad;  // [B, gamma, V] or null
};
hipError_t launch_tree_kl_loss(const TreeKlArgs& a, hipStream_t stream);

}  // namespace ubt
