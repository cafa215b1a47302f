// Softmax statistics and top-K candidate selection over the full vocabulary: one
// workgroup per row (the row code is in sweep.h).
//
// Method / Unigram Proposer, Eq. (ubtree-unigram), q_i = softmax(u_i), and "Candidate
// Sets": C_i = the K tokens of largest q_i, ranked on the logits with ties to the lower
// token id.
#include "sweep.h"
#include "sweep_big.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

// kBig: K > 16 (a tighter first threshold, a larger buffer with a running top K instead
// of the re-scan, and the workgroup-wide selection of sweep_big.h).
template <typename T, bool kAligned, bool kBig>
__global__ __launch_bounds__(kWave* kWaves, 4) void topk_row_kernel(const T* __restrict__ logits, int gamma,
                                                                    int64_t V, int64_t stride_b, int64_t stride_i,
                                                                    int K, int32_t* __restrict__ cand_ids,
                                                                    float* __restrict__ cand_logit,
                                                                    float* __restrict__ cand_logprob,
                                                                    float* __restrict__ lse) {
  const int64_t row = blockIdx.x;
  const int64_t b = row / gamma, i = row - b * gamma;
  const RowOut out{cand_ids, cand_logit, cand_logprob, lse, false};
  if constexpr (kBig) {
    __shared__ BigRowLds lds;
    sweep_row_big<T, kAligned>(lds, logits + b * stride_b + i * stride_i, V, K, row, out);
  } else {
    __shared__ RowLds lds;
    sweep_row<T, kAligned, kWaves, false>(lds, logits + b * stride_b + i * stride_i, V, K, row, out);
  }
}

template <typename T, bool kAligned>
void launch_typed(const void* logits, int B, int gamma, int64_t V, int64_t stride_b, int64_t stride_i, int K,
                  int32_t* cand_ids, float* cand_logit, float* cand_logprob, float* lse, hipStream_t stream) {
  const int64_t rows = static_cast<int64_t>(B) * gamma;
  if (K > 16)
    hipLaunchKernelGGL((topk_row_kernel<T, kAligned, true>), dim3(static_cast<unsigned>(rows)), dim3(kWave * kWaves),
                       0, stream, static_cast<const T*>(logits), gamma, V, stride_b, stride_i, K, cand_ids, cand_logit,
                       cand_logprob, lse);
  else
    hipLaunchKernelGGL((topk_row_kernel<T, kAligned, false>), dim3(static_cast<unsigned>(rows)), dim3(kWave * kWaves),
                       0, stream, static_cast<const T*>(logits), gamma, V, stride_b, stride_i, K, cand_ids, cand_logit,
                       cand_logprob, lse);
}

}  // namespace

hipError_t launch_topk(const void* logits, int dtype, bool aligned, int B, int gamma, int64_t V, int64_t stride_b,
                       int64_t stride_i, int K, int32_t* cand_ids, float* cand_logit, float* cand_logprob, float* lse,
                       hipStream_t stream) {
  if (dtype == 1) {
    if (aligned)
      launch_typed<uint16_t, true>(logits, B, gamma, V, stride_b, stride_i, K, cand_ids, cand_logit, cand_logprob,
                                   lse, stream);
    else
      launch_typed<uint16_t, false>(logits, B, gamma, V, stride_b, stride_i, K, cand_ids, cand_logit, cand_logprob,
                                    lse, stream);
  } else {
    if (aligned)
      launch_typed<float, true>(logits, B, gamma, V, stride_b, stride_i, K, cand_ids, cand_logit, cand_logprob, lse,
                                stream);
    else
      launch_typed<float, false>(logits, B, gamma, V, stride_b, stride_i, K, cand_ids, cand_logit, cand_logprob, lse,
                                 stream);
  }
  return hipGetLastError();
}

}  // namespace ubt
