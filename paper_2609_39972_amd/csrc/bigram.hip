// Selector scores and normalised transition log-probabilities for every adjacent
// candidate pair.
//
// Background, Eq. (dflash2-selector): delta_i(a,b) = (P(h_i) (.) phi(a))^T psi(b).
// Method / Parallel Computation, Eq. (ubtree-edge-matrix): all pairs of one depth form
// Delta_i = Phi_{i-1} diag(P(h_i)) Psi_i^T, with C_0 = {x_0} (one row at depth 1).
// Method / Depth Calibration, Eq. (ubtree-depth): s_i = alpha_i u_i(b) + lambda_i delta_i.
// Appendix A / Path Scores, Eq. (ubtree-path): log q^bi(b|a) = s_i(a,b) - log sum_v exp s_i(a,v).
// Without the normalisation (normalise = false) the same kernels write s_i itself: the
// edge scores of the unigram-plus-bigram scoring, given the candidates' log-probabilities
// in place of their logits.
//
// bf16 features: the rows of Phi and Psi are gathered straight into MFMA operand
// registers (v_mfma_f32_16x16x32_bf16, 16x16 output tiles).  K <= 16 (one tile) takes one
// wavefront per (sequence, depth).  Larger K takes one wavefront per row of output tiles:
// the waves split the r-contraction between them (wave w takes the 32-wide k-steps
// w, w + KT, ...), so each gathers a fraction of the rows' slots and all of its loads are
// in flight at once; the partial tiles then meet in LDS, each wave sums its own tile row
// over the waves in wave order and runs that row's epilogue (bigram_split_tile).  The
// gate is folded into the predecessor operand: g_k * phi_k(a) is exact in fp32 (two 8-bit
// significands) and is split into hi + lo bf16 parts, so the two MFMAs form every product
// g_k phi_k(a) psi_k(b) exactly and only the fp32 accumulation rounds.  The row
// log-softmax runs on the accumulator tile: a row of the tile lives in one aligned group
// of 16 lanes.  fp32 features use fp32 FMAs on the vector ALUs.
#include "bigram_tile.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

template <bool kNormalise>
__global__ __launch_bounds__(kWave) void bigram_bf16_kernel(const uint16_t* __restrict__ phi,
                                                            const uint16_t* __restrict__ psi,
                                                            const uint16_t* __restrict__ gate, int64_t V, int r,
                                                            const int32_t* __restrict__ anchor,
                                                            const int32_t* __restrict__ cand_ids,
                                                            const float* __restrict__ cand_logit, Scales sc,
                                                            int gamma, int K, float* __restrict__ delta,
                                                            float* __restrict__ logq) {
  const int64_t bi = blockIdx.x;  // b * gamma + i
  const int i = static_cast<int>(bi % gamma);
  const int64_t b = bi / gamma;
  bigram_tile_bf16<1, kNormalise>(phi, psi, gate + bi * r, V, r, i, K, anchor + b, i > 0 ? cand_ids + (bi - 1) * K : cand_ids, cand_ids + bi * K,
                       cand_logit + bi * K, sc.alpha[i], sc.lambda[i], delta ? delta + bi * K * K : nullptr,
                       logq + bi * K * K, nullptr, static_cast<int>(threadIdx.x));
}

template <int KT, bool kNormalise>  // output tiles per side, 16 (KT - 1) < K <= 16 KT; KT waves
__global__ __launch_bounds__(KT * kWave) __attribute__((amdgpu_waves_per_eu(2))) void bigram_bf16_split_kernel(
    const uint16_t* __restrict__ phi, const uint16_t* __restrict__ psi, const uint16_t* __restrict__ gate, int64_t V,
    int r, const int32_t* __restrict__ anchor, const int32_t* __restrict__ cand_ids,
    const float* __restrict__ cand_logit, Scales sc, int gamma, int K, float* __restrict__ delta,
    float* __restrict__ logq) {
  __shared__ f32x4 part[kSplitPartBytes<KT> / sizeof(f32x4)];
  const int lane = static_cast<int>(threadIdx.x) & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int64_t bi = blockIdx.x;  // b * gamma + i
  const int i = static_cast<int>(bi % gamma);
  const int64_t b = bi / gamma;
  bigram_split_tile<KT, kNormalise>(phi, psi, gate + bi * r, V, r, i, K, anchor + b,
                                    i > 0 ? cand_ids + (bi - 1) * K : cand_ids, cand_ids + bi * K, cand_logit + bi * K,
                                    sc.alpha[i], sc.lambda[i], delta ? delta + bi * K * K : nullptr, logq + bi * K * K,
                                    part, w, lane);
}

__global__ __launch_bounds__(kWave) void bigram_f32_kernel(const float* __restrict__ phi, const float* __restrict__ psi,
                                                           const float* __restrict__ gate, int64_t V, int r,
                                                           const int32_t* __restrict__ anchor,
                                                           const int32_t* __restrict__ cand_ids,
                                                           const float* __restrict__ cand_logit, Scales sc, int gamma,
                                                           int K, float* __restrict__ delta, float* __restrict__ logq,
                                                           int normalise) {
  __shared__ float s_delta[64 * 64];
  const int lane = threadIdx.x;
  const int64_t bi = blockIdx.x;
  const int i = static_cast<int>(bi % gamma);
  const int64_t b = bi / gamma;
  const int n_pred = (i == 0) ? 1 : K;
  const float* g = gate + bi * r;
  for (int pc = lane; pc < n_pred * K; pc += kWave) {
    const int a = pc / K, c = pc - a * K;
    const int64_t pa = clamp_id((i == 0) ? anchor[b] : cand_ids[(bi - 1) * K + a], V);
    const int64_t sb = clamp_id(cand_ids[bi * K + c], V);
    const float* pr = phi + pa * r;
    const float* sr = psi + sb * r;
    float d = 0.f;
    for (int k = 0; k < r; ++k) d = fmaf(g[k] * pr[k], sr[k], d);
    s_delta[pc] = d;
  }
  __syncthreads();
  const float al = sc.alpha[i], la = sc.lambda[i];
  float* dslab = delta ? delta + bi * K * K : nullptr;
  float* qslab = logq + bi * K * K;
  for (int a = lane; a < K; a += kWave) {
    if (a >= n_pred) {
      for (int c = 0; c < K; ++c) {
        if (dslab) dslab[a * K + c] = 0.f;
        qslab[a * K + c] = 0.f;
      }
      continue;
    }
    float norm = 0.f;
    if (normalise) {
      float m = neg_inf();
      for (int c = 0; c < K; ++c) m = fmaxf(m, fmaf(la, s_delta[a * K + c], al * cand_logit[bi * K + c]));
      float e = 0.f;
      for (int c = 0; c < K; ++c)
        e += __builtin_amdgcn_exp2f((fmaf(la, s_delta[a * K + c], al * cand_logit[bi * K + c]) - m) * kLog2e);
      norm = m + __builtin_amdgcn_logf(e) * kLn2;
    }
    for (int c = 0; c < K; ++c) {
      const float s = fmaf(la, s_delta[a * K + c], al * cand_logit[bi * K + c]);
      if (dslab) dslab[a * K + c] = s_delta[a * K + c];
      qslab[a * K + c] = normalise ? fminf(s - norm, 0.f) : s;
    }
  }
}

}  // namespace

hipError_t launch_bigram(const void* phi, const void* psi, const void* gate, int feat_dtype, int64_t V, int r,
                         const int32_t* anchor, const int32_t* cand_ids, const float* cand_logit, const Scales& scales,
                         int B, int gamma, int K, float* delta, float* logq, hipStream_t stream, bool normalise) {
  const dim3 grid(static_cast<unsigned>(static_cast<int64_t>(B) * gamma));
  const dim3 block(kWave);
  if (feat_dtype == 1) {
    const uint16_t* p = static_cast<const uint16_t*>(phi);
    const uint16_t* s = static_cast<const uint16_t*>(psi);
    const uint16_t* g = static_cast<const uint16_t*>(gate);
#define UBT_BIGRAM_ARGS p, s, g, V, r, anchor, cand_ids, cand_logit, scales, gamma, K, delta, logq
#define UBT_BIGRAM_K(NORM)                                                                                       \
  do {                                                                                                           \
    if (K <= 16)                                                                                                 \
      hipLaunchKernelGGL((bigram_bf16_kernel<NORM>), grid, dim3(kWave), 0, stream, UBT_BIGRAM_ARGS);             \
    else if (K <= 32)                                                                                            \
      hipLaunchKernelGGL((bigram_bf16_split_kernel<2, NORM>), grid, dim3(2 * kWave), 0, stream, UBT_BIGRAM_ARGS); \
    else                                                                                                         \
      hipLaunchKernelGGL((bigram_bf16_split_kernel<4, NORM>), grid, dim3(4 * kWave), 0, stream, UBT_BIGRAM_ARGS); \
  } while (0)
    if (normalise)
      UBT_BIGRAM_K(true);
    else
      UBT_BIGRAM_K(false);
#undef UBT_BIGRAM_K
#undef UBT_BIGRAM_ARGS
  } else {
    hipLaunchKernelGGL(bigram_f32_kernel, grid, block, 0, stream, static_cast<const float*>(phi),
                       static_cast<const float*>(psi), static_cast<const float*>(gate), V, r, anchor, cand_ids,
                       cand_logit, scales, gamma, K, delta, logq, normalise ? 1 : 0);
  }
  return hipGetLastError();
}

}  // namespace ubt
