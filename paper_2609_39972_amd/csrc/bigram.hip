// Selector scores and normalised transition log-probabilities for every adjacent
// candidate pair.
//
// Background, Eq. (dflash2-selector): delta_i(a,b) = (P(h_i) (.) phi(a))^T psi(b).
// Method / Parallel Computation, Eq. (ubtree-edge-matrix): all pairs of one depth form
// Delta_i = Phi_{i-1} diag(P(h_i)) Psi_i^T, with C_0 = {x_0} (one row at depth 1).
// Method / Depth Calibration, Eq. (ubtree-depth): s_i = alpha_i u_i(b) + lambda_i delta_i.
// Appendix A / Path Scores, Eq. (ubtree-path): log q^bi(b|a) = s_i(a,b) - log sum_v exp s_i(a,v).
//
// One wavefront per (sequence, depth).  bf16 features: the rows of Phi and Psi are
// gathered straight into MFMA operand registers (v_mfma_f32_16x16x32_bf16, 16x16 output
// tiles).  The gate is folded into the predecessor operand: g_k * phi_k(a) is exact in
// fp32 (two 8-bit significands) and is split into hi + lo bf16 parts, so the two MFMAs
// form every product g_k phi_k(a) psi_k(b) exactly and only the fp32 accumulation
// rounds.  The row log-softmax runs on the accumulator tile: a row of the tile lives in
// one aligned group of 16 lanes.  fp32 features use fp32 FMAs on the vector ALUs.
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Token ids come from device memory; out-of-range ids are clamped so a gather never
// leaves the tables (the scores of such a pair are then unspecified).
__device__ __forceinline__ int64_t clamp_id(int32_t id, int64_t V) { return id < 0 ? 0 : (id >= V ? V - 1 : id); }

// Predecessor operand for one k-slice: hi and lo bf16 parts of g_k * phi_k(a).
__device__ __forceinline__ void split_gated(u32x4 g, u32x4 p, u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t h2 = 0, l2 = 0;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int s = 16 * half;
      const float gv = __uint_as_float(((g[w] >> s) & 0xFFFFu) << 16);
      const float pv = __uint_as_float(((p[w] >> s) & 0xFFFFu) << 16);
      const float prod = gv * pv;                              // exact: 8-bit x 8-bit significands
      const uint32_t hb = __float_as_uint(prod) & 0xFFFF0000u;  // leading 8 significant bits
      const float rest = prod - __uint_as_float(hb);           // exact; at most 8 significant bits
      h2 |= (hb >> 16) << s;
      l2 |= (__float_as_uint(rest) >> 16) << s;
    }
    hi[w] = h2;
    lo[w] = l2;
  }
}

template <int KT>  // output tiles per side: K <= 16 * KT
__global__ __launch_bounds__(kWave) void bigram_bf16_kernel(const uint16_t* __restrict__ phi,
                                                            const uint16_t* __restrict__ psi,
                                                            const uint16_t* __restrict__ gate, int64_t V, int r,
                                                            const int32_t* __restrict__ anchor,
                                                            const int32_t* __restrict__ cand_ids,
                                                            const float* __restrict__ cand_logit, Scales sc,
                                                            int gamma, int K, float* __restrict__ delta,
                                                            float* __restrict__ logq) {
  const int lane = threadIdx.x;
  const int64_t bi = blockIdx.x;  // b * gamma + i
  const int i = static_cast<int>(bi % gamma);
  const int64_t b = bi / gamma;
  const int lr = lane & 15;  // operand row (A) / column (B) inside a tile
  const int kg = lane >> 4;  // k-slice group: slots 8*kg .. 8*kg+7 of each 32-wide step

  int64_t pred[KT], succ[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    const int a = 16 * t + lr;
    pred[t] = (i == 0) ? (a == 0 ? clamp_id(anchor[b], V) : -1) : (a < K ? clamp_id(cand_ids[(bi - 1) * K + a], V) : -1);
    const int c = 16 * t + lr;
    succ[t] = c < K ? clamp_id(cand_ids[bi * K + c], V) : -1;
  }

  f32x4 acc[KT][KT];
#pragma unroll
  for (int mt = 0; mt < KT; ++mt)
#pragma unroll
    for (int nt = 0; nt < KT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
  const uint16_t* g_row = gate + bi * r;
  for (int k0 = 8 * kg; k0 - 8 * kg < r; k0 += 32) {
    const bool in = k0 < r;
    const u32x4 g = in ? *reinterpret_cast<const u32x4*>(g_row + k0) : zero;
    u32x4 ahi[KT], alo[KT], bq[KT];
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      const u32x4 p = (in && pred[t] >= 0) ? *reinterpret_cast<const u32x4*>(phi + pred[t] * r + k0) : zero;
      split_gated(g, p, ahi[t], alo[t]);
      bq[t] = (in && succ[t] >= 0) ? *reinterpret_cast<const u32x4*>(psi + succ[t] * r + k0) : zero;
    }
#pragma unroll
    for (int mt = 0; mt < KT; ++mt)
#pragma unroll
      for (int nt = 0; nt < KT; ++nt) {
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ahi[mt]), as_bf16x8(bq[nt]), acc[mt][nt], 0, 0, 0);
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(alo[mt]), as_bf16x8(bq[nt]), acc[mt][nt], 0, 0, 0);
      }
  }

  // Epilogue.  acc[mt][nt][j] = delta(a, c) with a = 16 mt + 4 kg + j, c = 16 nt + lr.
  const float al = sc.alpha[i], la = sc.lambda[i];
  float au[KT];
#pragma unroll
  for (int nt = 0; nt < KT; ++nt) {
    const int c = 16 * nt + lr;
    au[nt] = c < K ? al * cand_logit[bi * K + c] : 0.f;
  }
  float* dslab = delta ? delta + bi * K * K : nullptr;
  float* qslab = logq + bi * K * K;
#pragma unroll
  for (int mt = 0; mt < KT; ++mt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int a = 16 * mt + 4 * kg + j;
      float s[KT];
      float m = neg_inf();
#pragma unroll
      for (int nt = 0; nt < KT; ++nt) {
        const int c = 16 * nt + lr;
        s[nt] = c < K ? fmaf(la, acc[mt][nt][j], au[nt]) : neg_inf();
        m = fmaxf(m, s[nt]);
      }
      m = group16_max(m);
      float e = 0.f;
#pragma unroll
      for (int nt = 0; nt < KT; ++nt) e += __builtin_amdgcn_exp2f((s[nt] - m) * kLog2e);
      e = group16_sum(e);
      const float norm = m + __builtin_amdgcn_logf(e) * kLn2;
      const bool real = (i == 0) ? a == 0 : a < K;
      if (a < K) {
#pragma unroll
        for (int nt = 0; nt < KT; ++nt) {
          const int c = 16 * nt + lr;
          if (c < K) {
            if (dslab) dslab[a * K + c] = real ? acc[mt][nt][j] : 0.f;
            qslab[a * K + c] = real ? fminf(s[nt] - norm, 0.f) : 0.f;
          }
        }
      }
    }
}

__global__ __launch_bounds__(kWave) void bigram_f32_kernel(const float* __restrict__ phi, const float* __restrict__ psi,
                                                           const float* __restrict__ gate, int64_t V, int r,
                                                           const int32_t* __restrict__ anchor,
                                                           const int32_t* __restrict__ cand_ids,
                                                           const float* __restrict__ cand_logit, Scales sc, int gamma,
                                                           int K, float* __restrict__ delta, float* __restrict__ logq) {
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
    float m = neg_inf();
    for (int c = 0; c < K; ++c) m = fmaxf(m, fmaf(la, s_delta[a * K + c], al * cand_logit[bi * K + c]));
    float e = 0.f;
    for (int c = 0; c < K; ++c)
      e += __builtin_amdgcn_exp2f((fmaf(la, s_delta[a * K + c], al * cand_logit[bi * K + c]) - m) * kLog2e);
    const float norm = m + __builtin_amdgcn_logf(e) * kLn2;
    for (int c = 0; c < K; ++c) {
      const float s = fmaf(la, s_delta[a * K + c], al * cand_logit[bi * K + c]);
      if (dslab) dslab[a * K + c] = s_delta[a * K + c];
      qslab[a * K + c] = fminf(s - norm, 0.f);
    }
  }
}

}  // namespace

hipError_t launch_bigram(const void* phi, const void* psi, const void* gate, int feat_dtype, int64_t V, int r,
                         const int32_t* anchor, const int32_t* cand_ids, const float* cand_logit, const Scales& scales,
                         int B, int gamma, int K, float* delta, float* logq, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(static_cast<int64_t>(B) * gamma));
  const dim3 block(kWave);
  if (feat_dtype == 1) {
    const uint16_t* p = static_cast<const uint16_t*>(phi);
    const uint16_t* s = static_cast<const uint16_t*>(psi);
    const uint16_t* g = static_cast<const uint16_t*>(gate);
    if (K <= 16)
      hipLaunchKernelGGL((bigram_bf16_kernel<1>), grid, block, 0, stream, p, s, g, V, r, anchor, cand_ids, cand_logit,
                         scales, gamma, K, delta, logq);
    else if (K <= 32)
      hipLaunchKernelGGL((bigram_bf16_kernel<2>), grid, block, 0, stream, p, s, g, V, r, anchor, cand_ids, cand_logit,
                         scales, gamma, K, delta, logq);
    else
      hipLaunchKernelGGL((bigram_bf16_kernel<4>), grid, block, 0, stream, p, s, g, V, r, anchor, cand_ids, cand_logit,
                         scales, gamma, K, delta, logq);
  } else {
    hipLaunchKernelGGL(bigram_f32_kernel, grid, block, 0, stream, static_cast<const float*>(phi),
                       static_cast<const float*>(psi), static_cast<const float*>(gate), V, r, anchor, cand_ids,
                       cand_logit, scales, gamma, K, delta, logq);
  }
  return hipGetLastError();
}

}  // namespace ubt
