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

// Table rows of the tile's operands: pred[t] is the predecessor of A-operand row
// a = 16 t + (lane & 15) (x_0 alone at i = 0), succ[t] the successor of B-operand column
// c = 16 t + (lane & 15); -1 past K (those operands are zero).
template <int KT>
__device__ __forceinline__ void tile_ids(int64_t V, int i, int K, const int32_t* anchor, const int32_t* pred_ids,
                                         const int32_t* succ_ids, int lane, int64_t (&pred)[KT],
                                         int64_t (&succ)[KT]) {
  const int lr = lane & 15;
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    const int a = 16 * t + lr;
    pred[t] = (i == 0) ? (a == 0 ? clamp_id(*anchor, V) : -1) : (a < K ? clamp_id(pred_ids[a], V) : -1);
    succ[t] = a < K ? clamp_id(succ_ids[a], V) : -1;
  }
}

// Operands of the 32-wide k-step starting at k = kb: lane group kg = lane >> 4 holds
// slots kb + 8 kg .. kb + 8 kg + 7 of the gate, of each predecessor row and of each
// successor row (zero past r and past K).
template <int KT>
__device__ __forceinline__ void load_step(const uint16_t* __restrict__ phi, const uint16_t* __restrict__ psi,
                                          const uint16_t* g_row, int r, int kb, const int64_t (&pred)[KT],
                                          const int64_t (&succ)[KT], int lane, u32x4& gq, u32x4 (&pq)[KT],
                                          u32x4 (&sq)[KT]) {
  const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
  const int k0 = kb + 8 * (lane >> 4);
  const bool in = k0 < r;
  gq = in ? *reinterpret_cast<const u32x4*>(g_row + k0) : zero;
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    pq[t] = (in && pred[t] >= 0) ? *reinterpret_cast<const u32x4*>(phi + pred[t] * r + k0) : zero;
    sq[t] = (in && succ[t] >= 0) ? *reinterpret_cast<const u32x4*>(psi + succ[t] * r + k0) : zero;
  }
}

// One k-step of every output tile: acc[mt][nt] += (hi + lo)(g phi)[rows of mt] psi[cols of nt]^T.
template <int KT>
__device__ __forceinline__ void mfma_step(u32x4 gq, const u32x4 (&pq)[KT], const u32x4 (&sq)[KT],
                                          f32x4 (&acc)[KT][KT]) {
  u32x4 ahi[KT], alo[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) split_gated(gq, pq[t], ahi[t], alo[t]);
#pragma unroll
  for (int mt = 0; mt < KT; ++mt)
#pragma unroll
    for (int nt = 0; nt < KT; ++nt) {
      acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ahi[mt]), as_bf16x8(sq[nt]), acc[mt][nt], 0, 0, 0);
      acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(alo[mt]), as_bf16x8(sq[nt]), acc[mt][nt], 0, 0, 0);
    }
}

// Unigram terms al * succ_logit[c] for the successor column c = 16 nt + (lane & 15) of
// each output tile column (0 past K).
template <int KT>
__device__ __forceinline__ void succ_terms(const float* succ_logit, float al, int K, int lane, float (&au)[KT]) {
#pragma unroll
  for (int nt = 0; nt < KT; ++nt) {
    const int c = 16 * nt + (lane & 15);
    au[nt] = c < K ? al * succ_logit[c] : 0.f;
  }
}

// Epilogue of one row of output tiles: accr[nt][j] = delta(a, c) with a = 16 mt + 4 kg + j,
// c = 16 nt + (lane & 15), kg = lane >> 4.  Forms s = al u + la delta and, with
// kNormalise, the log-softmax over the K successors of each row (a row lives in one
// aligned group of 16 lanes), then writes rows a < K.
// kCoherent: qslab is written with agent-scope stores, which reach the device-coherent
// level, for a reader in another workgroup of the same launch.
template <int KT, bool kNormalise, bool kCoherent = false>
__device__ __forceinline__ void tile_rows_out(const f32x4 (&accr)[KT], int mt, int i, int K, const float (&au)[KT],
                                              float la, float* dslab, float* qslab, float* qslab2, int lane) {
  const int lr = lane & 15, kg = lane >> 4;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int a = 16 * mt + 4 * kg + j;
    float s[KT];
    float m = neg_inf();
#pragma unroll
    for (int nt = 0; nt < KT; ++nt) {
      const int c = 16 * nt + lr;
      s[nt] = c < K ? fmaf(la, accr[nt][j], au[nt]) : neg_inf();
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
          if (dslab) dslab[a * K + c] = real ? accr[nt][j] : 0.f;
          if constexpr (kCoherent)
            __hip_atomic_store(reinterpret_cast<uint32_t*>(qslab + a * K + c), __float_as_uint(q), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
          else
            qslab[a * K + c] = q;
          if (qslab2) qslab2[a * K + c] = q;
        }
      }
    }
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
  int64_t pred[KT], succ[KT];
  tile_ids<KT>(V, i, K, anchor, pred_ids, succ_ids, lane, pred, succ);

  f32x4 acc[KT][KT];
#pragma unroll
  for (int mt = 0; mt < KT; ++mt)
#pragma unroll
    for (int nt = 0; nt < KT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // The k range is walked in 32-wide steps, ceil(r / 32) of them, in order; the operands
  // of kSteps consecutive steps are gathered together so their loads overlap.
  constexpr int kSteps = 4;
  for (int kb = 0; kb < r; kb += 32 * kSteps) {
    u32x4 gq[kSteps], pq[kSteps][KT], sq[kSteps][KT];
#pragma unroll
    for (int st = 0; st < kSteps; ++st) load_step<KT>(phi, psi, g_row, r, kb + 32 * st, pred, succ, lane, gq[st], pq[st], sq[st]);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (kb + 32 * st >= r) break;  // wave-uniform: no step past ceil(r / 32)
      mfma_step<KT>(gq[st], pq[st], sq[st], acc);
    }
  }

  float au[KT];
  succ_terms<KT>(succ_logit, al, K, lane, au);
#pragma unroll
  for (int mt = 0; mt < KT; ++mt) tile_rows_out<KT, kNormalise>(acc[mt], mt, i, K, au, la, dslab, qslab, qslab2, lane);
}

// K > 16: the same scores on KT waves of one workgroup, one wave per row of output tiles.
// The waves split the r-contraction between them (wave w takes the 32-wide k-steps
// w, w + KT, ...), so each gathers a fraction of every row and all of its loads are in
// flight at once; the partial tiles then meet in `part` (workgroup LDS of
// kSplitPartBytes<KT> bytes), and wave w sums tile row w over the waves in wave order and
// runs that row's epilogue.  All KT waves of the workgroup must call it (it holds one
// workgroup barrier); w is the caller's wave index.
template <int KT>
constexpr size_t kSplitPartBytes = static_cast<size_t>(KT) * (KT - 1) * KT * kWave * sizeof(f32x4);

template <int KT, bool kNormalise, bool kCoherent = false>
__device__ __forceinline__ void bigram_split_tile(const uint16_t* __restrict__ phi, const uint16_t* __restrict__ psi,
                                                  const uint16_t* g_row, int64_t V, int r, int i, int K,
                                                  const int32_t* anchor, const int32_t* pred_ids,
                                                  const int32_t* succ_ids, const float* succ_logit, float al,
                                                  float la, float* dslab, float* qslab, f32x4* part, int w,
                                                  int lane) {
  // part[((v (KT - 1) + s) KT + nt) 64 + lane]: wave v's partial of tile (mt, nt) for the
  // s-th tile row mt != v.
  int64_t pred[KT], succ[KT];
  tile_ids<KT>(V, i, K, anchor, pred_ids, succ_ids, lane, pred, succ);
  f32x4 acc[KT][KT];
#pragma unroll
  for (int mt = 0; mt < KT; ++mt)
#pragma unroll
    for (int nt = 0; nt < KT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // This wave's k-steps w, w + KT, ..., kSteps of them gathered together.
  const int n_steps = (r + 31) / 32;
  constexpr int kSteps = 2;
  for (int s0 = w; s0 < n_steps; s0 += KT * kSteps) {
    u32x4 gq[kSteps], pq[kSteps][KT], sq[kSteps][KT];
#pragma unroll
    for (int st = 0; st < kSteps; ++st)
      load_step<KT>(phi, psi, g_row, r, 32 * (s0 + KT * st), pred, succ, lane, gq[st], pq[st], sq[st]);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (s0 + KT * st >= n_steps) break;  // wave-uniform
      mfma_step<KT>(gq[st], pq[st], sq[st], acc);
    }
  }

  // Hand over the tile rows the other waves finish; keep this wave's own row.
  f32x4 own[KT];
#pragma unroll
  for (int mt = 0; mt < KT; ++mt) {
    if (mt == w) {
#pragma unroll
      for (int nt = 0; nt < KT; ++nt) own[nt] = acc[mt][nt];
    } else {
      const int slot = mt < w ? mt : mt - 1;
#pragma unroll
      for (int nt = 0; nt < KT; ++nt) part[((w * (KT - 1) + slot) * KT + nt) * kWave + lane] = acc[mt][nt];
    }
  }
  __syncthreads();
  f32x4 row[KT];
#pragma unroll
  for (int nt = 0; nt < KT; ++nt) row[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int v = 0; v < KT; ++v) {
    if (v == w) {
#pragma unroll
      for (int nt = 0; nt < KT; ++nt) row[nt] += own[nt];
    } else {
      const int slot = w < v ? w : w - 1;
#pragma unroll
      for (int nt = 0; nt < KT; ++nt) row[nt] += part[((v * (KT - 1) + slot) * KT + nt) * kWave + lane];
    }
  }

  float au[KT];
  succ_terms<KT>(succ_logit, al, K, lane, au);
  tile_rows_out<KT, kNormalise, kCoherent>(row, w, i, K, au, la, dslab, qslab, nullptr, lane);
}

}  // namespace ubt
