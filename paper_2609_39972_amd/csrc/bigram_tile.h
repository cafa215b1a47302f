// One tile of selector scores: Delta_i, s_i and log q^bi for one (sequence, position),
// computed by one wavefront on the matrix cores.  Shared by the standalone selector
// kernel and the fused selector + tree-search kernel, so both produce the same bits.
//
// Background, Eq. (dflash2-selector): delta_i(a,b) = (P(h_i) (.) phi(a))^T psi(b).
// Method / Parallel Computation, Eq. (ubtree-edge-matrix): all pairs of one depth form
// Delta_i = Phi_{i-1} diag(P(h_i)) Psi_i^T, with C_0 = {x_0} (one row at depth 1).
// Method / Depth Calibration, Eq. (ubtree-depth): s_i = alpha_i u_i(b) + lambda_i delta_i.
// Appendix A / Path Scores, Eq. (ubtree-path): log q^bi(b|a) = s_i(a,b) - log sum_v exp s_i(a,v).
//
// The rows of Phi and Psi are gathered straight into MFMA operand registers
// (v_mfma_f32_16x16x32_bf16, 16x16 output tiles).  The gate is folded into the
// predecessor operand: g_k * phi_k(a) is exact in fp32 (two 8-bit significands) and is
// split into hi + lo bf16 parts, so the two MFMAs form every product g_k phi_k(a)
// psi_k(b) exactly and only the fp32 accumulation rounds.  The row log-softmax runs on
// the accumulator tile: a row of the tile lives in one aligned group of 16 lanes.
#pragma once

#include "ubt_device.h"

namespace ubt {

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

// Scores of position i (depth i + 1) of one sequence.  anchor points at x_0 (read at
// i = 0 only); pred_ids = C_{i-1} (read at i > 0 only); succ_ids / succ_logit = C_i and
// its logits; g_row = P(h_i).  Writes delta (if dslab) and log q^bi to qslab and, if
// given, qslab2, each [K][K] indexed [a][c].  All 64 lanes of the wave must call it.
// kNormalise = false writes s_i(a, c) = al * succ_logit[c] + la * delta(a, c) itself,
// with no normalisation over the successors (edge scores of the unigram-plus-bigram
// scoring, where succ_logit holds the candidates' log-probabilities).
template <int KT, bool kNormalise = true>  // output tiles per side: K <= 16 * KT
__device__ __forceinline__ void bigram_tile_bf16(const uint16_t* __restrict__ phi, const uint16_t* __restrict__ psi,
                                                 const uint16_t* g_row, int64_t V, int r, int i, int K,
                                                 const int32_t* anchor, const int32_t* pred_ids,
                                                 const int32_t* succ_ids, const float* succ_logit, float al,
                                                 float la, float* dslab, float* qslab, float* qslab2, int lane) {
  const int lr = lane & 15;  // operand row (A) / column (B) inside a tile
  const int kg = lane >> 4;  // k-slice group: slots 8*kg .. 8*kg+7 of each 32-wide step

  int64_t pred[KT], succ[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    const int a = 16 * t + lr;
    pred[t] = (i == 0) ? (a == 0 ? clamp_id(*anchor, V) : -1) : (a < K ? clamp_id(pred_ids[a], V) : -1);
    const int c = 16 * t + lr;
    succ[t] = c < K ? clamp_id(succ_ids[c], V) : -1;
  }

  f32x4 acc[KT][KT];
#pragma unroll
  for (int mt = 0; mt < KT; ++mt)
#pragma unroll
    for (int nt = 0; nt < KT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // The k range is walked in 32-wide steps, ceil(r / 32) of them, in order; the operands
  // of kSteps consecutive steps are gathered together so their loads overlap.
  constexpr int kSteps = 4;
  const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
  for (int kb = 0; kb < r; kb += 32 * kSteps) {
    u32x4 gq[kSteps], pq[kSteps][KT], sq[kSteps][KT];
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      const int k0 = kb + 32 * st + 8 * kg;
      const bool in = k0 < r;
      gq[st] = in ? *reinterpret_cast<const u32x4*>(g_row + k0) : zero;
#pragma unroll
      for (int t = 0; t < KT; ++t) {
        pq[st][t] = (in && pred[t] >= 0) ? *reinterpret_cast<const u32x4*>(phi + pred[t] * r + k0) : zero;
        sq[st][t] = (in && succ[t] >= 0) ? *reinterpret_cast<const u32x4*>(psi + succ[t] * r + k0) : zero;
      }
    }
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (kb + 32 * st >= r) break;  // wave-uniform: no step past ceil(r / 32)
      u32x4 ahi[KT], alo[KT];
#pragma unroll
      for (int t = 0; t < KT; ++t) split_gated(gq[st], pq[st][t], ahi[t], alo[t]);
#pragma unroll
      for (int mt = 0; mt < KT; ++mt)
#pragma unroll
        for (int nt = 0; nt < KT; ++nt) {
          acc[mt][nt] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ahi[mt]), as_bf16x8(sq[st][nt]), acc[mt][nt], 0, 0, 0);
          acc[mt][nt] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(alo[mt]), as_bf16x8(sq[st][nt]), acc[mt][nt], 0, 0, 0);
        }
    }
  }

  // Epilogue.  acc[mt][nt][j] = delta(a, c) with a = 16 mt + 4 kg + j, c = 16 nt + lr.
  float au[KT];
#pragma unroll
  for (int nt = 0; nt < KT; ++nt) {
    const int c = 16 * nt + lr;
    au[nt] = c < K ? al * succ_logit[c] : 0.f;
  }
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
      float norm = 0.f;
      if (kNormalise) {
        m = group16_max(m);
        float e = 0.f;
#pragma unroll
        for (int nt = 0; nt < KT; ++nt) e += __builtin_amdgcn_exp2f((s[nt] - m) * kLog2e);
        e = group16_sum(e);
        norm = m + __builtin_amdgcn_logf(e) * kLn2;
      }
      const bool real = (i == 0) ? a == 0 : a < K;
      if (a < K) {
#pragma unroll
        for (int nt = 0; nt < KT; ++nt) {
          const int c = 16 * nt + lr;
          if (c < K) {
            const float q = real ? (kNormalise ? fminf(s[nt] - norm, 0.f) : s[nt]) : 0.f;
            if (dslab) dslab[a * K + c] = real ? acc[mt][nt][j] : 0.f;
            qslab[a * K + c] = q;
            if (qslab2) qslab2[a * K + c] = q;
          }
        }
      }
    }
}

}  // namespace ubt
