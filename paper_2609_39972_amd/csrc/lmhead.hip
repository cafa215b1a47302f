// The LM-head projection fused with the softmax statistics and the candidate sets: the
// logits never reach device memory.
//
// Background, "DFlash & DFlash 2": the proposer's hidden state h_i is mapped to its
// logits u_i by the frozen target LM head, u_i = W_lm h_i.  Method / Unigram Proposer,
// Eq. (ubtree-unigram) and "Candidate Sets": LSE_i, and C_i = the K largest u_i(v),
// ordered (u desc, id asc).
//
// For a drafting block (up to 16 rows of h per group) the projection reads every row of
// W_lm once and does 2 * 16 flops per weight element, so it is bound by the bandwidth of
// streaming W_lm, not by the matrix cores.
//
// Stream kernel: persistent workgroups of 8 waves.  Wave t of the grid takes the 16-row
// vocabulary tiles t, t + T, ... (T = waves in the grid); for each tile it runs the d / 32
// steps of v_mfma_f32_16x16x32_bf16 with 16 rows of h as the A operand and the tile's 16
// rows of W_lm as the B operand, with up to 16 k-steps of loads in flight.  Each tile's
// 16 x 16 logits go to the workgroup's LDS: per row of h, one slot per vocabulary row the
// workgroup covers, in id order.  After the last tile each wave takes up to two rows of h:
// their maximum and sum of exp(u - max), and their exact top K under (logit desc, id asc)
// by the ballot radix selection, written as (order key, id) pairs with the K-th one's
// 64-bit order value.
//
// Merge kernel, one workgroup per row of h: LSE from the workgroups' (max, sum) pairs in a
// fixed order; then the candidates.  Every workgroup's K-th order value is a lower bound
// of the row's K-th (the workgroup holds K entries at or above it), and every entry of the
// row's top K is in its own workgroup's top K, so the entries at or above the largest of
// these bounds hold the row's top K.  An 8-bit radix selection over their 64-bit order
// values finds the K-th, and the K entries at or above it are ranked by counting.
#include <type_traits>

#include "bigram_tile.h"
#include "search.h"

namespace ubt {
namespace {

constexpr int kLmWaves = 8;
constexpr int kLmRows = 16;       // rows of h per group (one MFMA tile)
constexpr int kLmMaxRounds = 16;  // tiles per wave: LDS holds 16 x (rounds * 128) logits
constexpr int kLmRowPad = 4;      // LDS row padding (floats): spreads a tile's 4 row groups over the banks
constexpr int kLmMergeThreads = 256;
constexpr int kLmStageWords = 2 * (64 + 2);  // per-wave selection stage: two rows of K + 2 (K <= 64)

struct LmArgs {
  const uint16_t* h;  // [M, d] bf16
  const uint16_t* w;  // [V, d] bf16
  int M, d, K;
  int64_t V;
  int n_tiles;  // ceil(V / 16)
  int rounds;   // ceil(n_tiles / (gridDim.x * kLmWaves))
  float2* part_ms;   // [groups][G][16] (max, sum of exp(u - max)); max = -inf: nothing
  uint2* part_cand;  // [groups][G][16][K] (order key, id) sorted by (logit desc, id asc); key 0 = none
  int32_t* cand_ids;
  float* cand_logit;
  float* cand_logprob;
  float* lse;
};

// 64-bit order of (logit key, id): larger is better under (logit desc, id asc).
__device__ __forceinline__ uint64_t lm_order(uint32_t key, uint32_t id) {
  return (static_cast<uint64_t>(key) << 32) | static_cast<uint32_t>(~id);
}

// One row of a workgroup's logits during the per-row selection (registers of one wave).
template <int NR>
struct RowSel {
  float x[NR];
  uint32_t key[NR];  // order key, 0 for an empty slot
  float mx, se;      // maximum and sum of exp(u - max)
  int need;          // entries to take: min(K, live entries)
  uint32_t thr;      // threshold key
  bool exact;        // exactly `need` live keys are >= thr (else ties at thr by slot)
};

template <int NR>
__device__ __forceinline__ void row_load(RowSel<NR>& R, const float* row, int nslot, int lane, bool live, int K) {
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int s = r * kWave + lane;
    R.x[r] = live && s < nslot ? row[s] : neg_inf();
    R.key[r] = R.x[r] == neg_inf() ? 0u : f32_key(R.x[r]);
  }
  float mx = neg_inf();
#pragma unroll
  for (int r = 0; r < NR; ++r) mx = fmaxf(mx, R.x[r]);
  R.mx = wave_max(mx);
  float se = 0.f;
#pragma unroll
  for (int r = 0; r < NR; ++r) se += R.key[r] != 0u ? __builtin_amdgcn_exp2f((R.x[r] - R.mx) * kLog2e) : 0.f;
  R.se = wave_sum(se);
  int n_live = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) n_live += popc(ballot(R.key[r] != 0u));
  R.need = n_live < K ? n_live : K;
  R.thr = 1u;  // every live key is >= 1
  R.exact = true;
}

// Search state of the need-th largest key of a row: a ballot radix search over the bits
// below the common prefix of the largest key and a lower bound of the answer, stopping at
// the first exact split.  The lower bound is the smallest per-lane maximum when at least
// `need` lanes hold a key (each of those lanes has a key at or above it), else the
// smallest key.
struct RadixState {
  uint32_t m, t, cand;
  int cnt;
};

template <int NR>
__device__ __forceinline__ RadixState radix_begin(RowSel<NR>& R) {
  RadixState S{0u, 0u, 0u, 0};
  uint32_t hi = 0u, lo = ~0u;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    hi = max(hi, R.key[r]);
    lo = min(lo, R.key[r] != 0u ? R.key[r] : ~0u);
  }
  int n_live = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) n_live += popc(ballot(R.key[r] != 0u));
  if (n_live <= R.need) return S;  // every live key is taken
  const uint32_t kmax = wave_umax(hi);
  uint32_t kmin = wave_umin(lo);
  const int lanes = popc(ballot(hi != 0u));
  if (lanes >= R.need) kmin = max(kmin, wave_umin(hi != 0u ? hi : ~0u));
  R.exact = false;
  if (kmax == kmin) {
    R.thr = kmax;
    return S;
  }
  S.m = 0x80000000u >> __clz(kmax ^ kmin);
  S.t = kmax & ~(S.m | (S.m - 1u));
  return S;
}

template <int NR>
__device__ __forceinline__ void radix_step(const RowSel<NR>& R, RadixState& S) {
  S.cand = S.t | S.m;
  int cnt = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) cnt += popc(ballot(R.key[r] >= S.cand));  // empty slots (0) never count
  S.cnt = cnt;
  S.t = cnt > R.need ? S.cand : S.t;
  S.m = radix_next(S.m, cnt, R.need, 0u);
}

template <int NR>
__device__ __forceinline__ void radix_end(RowSel<NR>& R, const RadixState& S) {
  if (R.exact || R.thr != 1u) return;  // no search ran (everything taken, or all keys equal)
  if (S.cnt == R.need) {
    R.thr = S.cand;
    R.exact = true;
  } else {
    R.thr = S.t;
  }
}

// The selected entries' order values to stage[0..need) in slot order, then stage[need] =
// stage[need + 1] = 0 (below every entry).
template <int NR, class SlotId>
__device__ __forceinline__ void row_compact(const RowSel<NR>& R, uint64_t* stage, int lane, SlotId slot_id) {
  int left = 0;
  if (!R.exact) {
    int above = 0;
#pragma unroll
    for (int r = 0; r < NR; ++r) above += popc(ballot(R.key[r] > R.thr));
    left = R.need - above;
  }
  int pos = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    uint64_t msk = ballot(R.key[r] >= R.thr);
    if (!R.exact) {
      const uint64_t eq = ballot(R.key[r] == R.thr);
      msk = ballot(R.key[r] > R.thr) | ballot(lane_in(eq) && static_cast<int>(lanes_below(eq)) < left);
      const int te = popc(eq);
      left -= te < left ? te : left;
    }
    if (lane_in(msk)) stage[pos + static_cast<int>(lanes_below(msk))] = lm_order(R.key[r], slot_id(r * kWave + lane));
    pos += popc(msk);
  }
  if (lane < 2) stage[R.need + lane] = 0ull;
}

// Lane < need: its staged entry and its rank (entries above it), read two at a time.
__device__ __forceinline__ int stage_rank(const uint64_t* stage, int need, uint64_t mine) {
  const ulonglong2* p = reinterpret_cast<const ulonglong2*>(stage);
  int rank = 0;
  for (int j = 0; j < (need + 1) / 2; ++j) {
    const ulonglong2 o = p[j];
    rank += (o.x > mine ? 1 : 0) + (o.y > mine ? 1 : 0);
  }
  return rank;
}

// Per row m < Mg of the group (wave w takes rows w and w + 8, interleaved so that their
// dependent steps overlap): the maximum and sum of exp(u - max) of the workgroup's logits
// vals[m][0..nslot), and their exact top K under (logit desc, id asc), written as (order
// key, id) pairs in that order.  slot_id(s) is the vocabulary id of slot s and must
// increase with s, so (key desc, slot asc) is (logit desc, id asc).  Empty slots hold
// -inf.  stage: this wave's LDS scratch of 2 (K + 2) 64-bit words, 16-byte aligned.  NR:
// registers per lane for a row (nslot <= 64 NR).
template <int NR, class SlotId>
__device__ __forceinline__ void emit_rows(const LmArgs& a, const float* vals, int rstride, int nslot, int Mg, int w,
                                          int lane, int64_t pbase, uint64_t* stage, SlotId slot_id) {
  static_assert(kLmRows <= 2 * kLmWaves, "two rows per wave");
  const int K = a.K;
  const int m0 = w, m1 = w + kLmWaves;
  if (m0 >= Mg) return;
  const bool has1 = m1 < Mg;
  RowSel<NR> R0, R1;
  row_load<NR>(R0, vals + m0 * rstride, nslot, lane, true, K);
  row_load<NR>(R1, vals + (has1 ? m1 : m0) * rstride, nslot, lane, has1, K);
  RadixState S0 = radix_begin<NR>(R0), S1 = radix_begin<NR>(R1);
  while (S0.m != 0u || S1.m != 0u) {
    if (S0.m != 0u) radix_step<NR>(R0, S0);
    if (S1.m != 0u) radix_step<NR>(R1, S1);
  }
  radix_end<NR>(R0, S0);
  radix_end<NR>(R1, S1);
  const int st1 = (K + 3) & ~1;  // even, so the second stage stays 16-byte aligned
  uint64_t* stage0 = stage;
  uint64_t* stage1 = stage + st1;
  row_compact<NR>(R0, stage0, lane, slot_id);
  row_compact<NR>(R1, stage1, lane, slot_id);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
  const uint64_t mine0 = lane < R0.need ? stage0[lane] : 0ull;
  const uint64_t mine1 = lane < R1.need ? stage1[lane] : 0ull;
  const int rank0 = lane < R0.need ? stage_rank(stage0, R0.need, mine0) : 0;
  const int rank1 = lane < R1.need ? stage_rank(stage1, R1.need, mine1) : 0;
  auto store = [&](int m, const RowSel<NR>& R, uint64_t mine, int rank) {
    const int64_t pidx = pbase + m;
    uint2* out = a.part_cand + pidx * K;
    if (lane < R.need) out[rank] = make_uint2(static_cast<uint32_t>(mine >> 32), ~static_cast<uint32_t>(mine));
    for (int e = R.need + lane; e < K; e += kWave) out[e] = make_uint2(0u, 0u);
    if (lane == 0) a.part_ms[pidx] = make_float2(R.mx, R.se);
  };
  store(m0, R0, mine0, rank0);
  if (has1) store(m1, R1, mine1, rank1);
}

// P: k-steps per chunk of loads in flight (divides d / 32); NR: registers per lane holding
// one row's slots (2 * rounds <= NR).
template <int P, int NR>
__global__ __launch_bounds__(kLmWaves* kWave) void lm_head_stream_kernel(LmArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* vals = reinterpret_cast<float*>(smem_raw);  // [16][rstride]
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int lr = lane & 15, kg = lane >> 4;
  const int G = static_cast<int>(gridDim.x);
  const int g = static_cast<int>(blockIdx.x);
  const int grp = static_cast<int>(blockIdx.y);
  const int row0 = grp * kLmRows;
  const int Mg = a.M - row0 < kLmRows ? a.M - row0 : kLmRows;
  const int nslot = a.rounds * kLmWaves * 16;
  const int rstride = nslot + kLmRowPad;
  for (int e = static_cast<int>(threadIdx.x); e < kLmRows * rstride; e += static_cast<int>(blockDim.x))
    vals[e] = neg_inf();
  __syncthreads();

  // ---- streaming: this wave's tiles, d / 32 k-steps each --------------------------------
  // Steps run in chunks of P (P divides d / 32); the loads of the next chunk (of this tile,
  // else of the next tile) are issued as the current chunk's MFMAs consume theirs, so P
  // k-steps of loads stay in flight.  After the last chunk the wave re-reads its last
  // chunk instead (a valid address, results unused), so the loop body has no branch.
  const int d = a.d, S = d / 32;
  const int wave_g = g * kLmWaves + w, stride = G * kLmWaves;
  const int ntw = wave_g < a.n_tiles ? (a.n_tiles - wave_g + stride - 1) / stride : 0;
  // Lanes past the group's rows of h, or past the last vocabulary row, read a valid row
  // instead: their accumulator entries are never stored.
  const uint16_t* hp = a.h + static_cast<int64_t>(row0 + (lr < Mg ? lr : Mg - 1)) * d + 8 * kg;
  auto tile_row = [&](int j) {
    int64_t v = (static_cast<int64_t>(wave_g) + static_cast<int64_t>(j) * stride) * 16 + lr;
    if (v >= a.V) v = a.V - 1;
    return a.w + v * d + 8 * kg;
  };
  if (ntw > 0) {
    u32x4 ra[P], rb[P];
    const uint16_t* wt = tile_row(0);
#pragma unroll
    for (int u = 0; u < P; ++u) {
      ra[u] = *reinterpret_cast<const u32x4*>(hp + 32 * u);
      rb[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wt + 32 * u));
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int t = 0; t < ntw; ++t) {
      const uint16_t* wnext = tile_row(t + 1 < ntw ? t + 1 : t);
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int c = 0; c < S; c += P) {
        const bool last = c + P == S;
        const uint16_t* wn = last ? (t + 1 < ntw ? wnext : wt + c * 32) : wt + (c + P) * 32;
        const uint16_t* hn = hp + (last ? (t + 1 < ntw ? 0 : c * 32) : (c + P) * 32);
#pragma unroll
        for (int u = 0; u < P; ++u) {
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ra[u]), as_bf16x8(rb[u]), acc, 0, 0, 0);
          ra[u] = *reinterpret_cast<const u32x4*>(hn + 32 * u);
          rb[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wn + 32 * u));
          // Keep loads in consumption order, so each MFMA waits only for its own operands.
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // Tile done: acc[j] = u(row 4 kg + j of the group, vocabulary row 16 tile + lr).
      const int64_t v = (static_cast<int64_t>(wave_g) + static_cast<int64_t>(t) * stride) * 16 + lr;
      const int slot = (t * kLmWaves + w) * 16 + lr;
      if (v < a.V) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (4 * kg + j < Mg) vals[(4 * kg + j) * rstride + slot] = acc[j];
      }
      wt = wnext;
    }
  }
  __syncthreads();
  // Slot s = (round * 8 + wave) * 16 + column holds vocabulary id
  // ((g * 8 + wave) + round * T) * 16 + column.
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem_raw + kLmRows * rstride * sizeof(float)) + w * kLmStageWords;
  emit_rows<NR>(a, vals, rstride, nslot, Mg, w, lane, (static_cast<int64_t>(grp) * G + g) * kLmRows, stage, [&](int s) {
    const int col = s & 15, wv = (s >> 4) & (kLmWaves - 1), round = s >> 7;
    return static_cast<uint32_t>((static_cast<int64_t>(g) * kLmWaves + wv + static_cast<int64_t>(round) * stride) * 16 +
                                 col);
  });
}

constexpr int kLmTRow = 144;  // bytes per row of a wave's transpose buffer: 128 + 16 (bank spread)

struct SplitLayout {
  uint32_t vals, tbuf, red, total;
};

__host__ __device__ inline SplitLayout split_layout(int rstride) {
  SplitLayout L{};
  L.vals = 0;
  L.tbuf = static_cast<uint32_t>(kLmRows * rstride * 4);
  L.red = L.tbuf + kLmWaves * kLmRows * kLmTRow;
  L.total = L.red + 2 * kLmWaves * 256 * 4;
  return L;
}

// Split kernel (d = 256 * SW, SW even): the 8 waves of a workgroup take the same 16-row
// vocabulary tile at once, wave w the k-slice [w d/8, (w+1) d/8), so each wave holds its
// slice of h as MFMA A operands in registers for the whole launch and h is read once.
// Each load instruction reads 128 contiguous bytes of 8 head rows (8 lanes per row, whole
// cache lines); the wave's LDS buffer turns two such loads (16 rows x 64 k) into the B
// operands of two MFMA steps.  The loads of the next tile are issued as the current one's
// registers are freed, so a whole tile slice (SW loads) stays in flight per wave (the last tile
// issues none).  After
// each tile the 8 partial 16 x 16 products are summed in wave order through LDS.
template <int SW, int NR>
__global__ __launch_bounds__(kLmWaves* kWave) void lm_head_split_kernel(LmArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int lr = lane & 15, kg = lane >> 4;
  const int G = static_cast<int>(gridDim.x);
  const int g = static_cast<int>(blockIdx.x);
  const int grp = static_cast<int>(blockIdx.y);
  const int row0 = grp * kLmRows;
  const int Mg = a.M - row0 < kLmRows ? a.M - row0 : kLmRows;
  const int nslot = a.rounds * 16;
  const int rstride = nslot + kLmRowPad;
  const SplitLayout L = split_layout(rstride);
  float* vals = reinterpret_cast<float*>(smem_raw + L.vals);  // [16][rstride]
  unsigned char* tb = smem_raw + L.tbuf + w * kLmRows * kLmTRow;
  float* red = reinterpret_cast<float*>(smem_raw + L.red);  // [2][8 waves][256]
  for (int e = static_cast<int>(threadIdx.x); e < kLmRows * rstride; e += static_cast<int>(blockDim.x))
    vals[e] = neg_inf();

  constexpr int kSeg = SW / 2;  // 128-byte segments per row of the slice
  const int d = a.d;
  const int ks0 = w * SW * 32;  // first k of this wave's slice
  // A operands: step s takes k = ks0 + 32 s + 8 kg .. + 8 of row lr of the group (rows past
  // the group read its last row; their results are never stored).
  u32x4 A[SW];
  {
    const uint16_t* hp = a.h + static_cast<int64_t>(row0 + (lr < Mg ? lr : Mg - 1)) * d + ks0 + 8 * kg;
#pragma unroll
    for (int s2 = 0; s2 < SW; ++s2) A[s2] = *reinterpret_cast<const u32x4*>(hp + 32 * s2);
  }
  // Loads: segment c of tile j, row group rg: lane reads row 16 t_j + 8 rg + lane / 8 at
  // bytes 2 ks0 + 128 c + 16 (lane % 8) (rows past V read row V - 1).
  const int ntw = g < a.n_tiles ? (a.n_tiles - g + G - 1) / G : 0;
  const int lrow = lane >> 3, lbyte = (lane & 7) * 16;
  auto row_ptr = [&](int j, int rg) {
    int64_t v = static_cast<int64_t>(g + j * G) * 16 + rg * 8 + lrow;
    if (v >= a.V) v = a.V - 1;
    return reinterpret_cast<const unsigned char*>(a.w) + v * (2 * static_cast<int64_t>(d)) + 2 * ks0 + lbyte;
  };
  u32x4 R[SW];  // R[2c + rg]: segment c, row group rg
  if (ntw > 0) {
    const unsigned char* p0 = row_ptr(0, 0);
    const unsigned char* p1 = row_ptr(0, 1);
#pragma unroll
    for (int c = 0; c < kSeg; ++c) {
      R[2 * c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p0 + 128 * c));
      R[2 * c + 1] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p1 + 128 * c));
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // Transpose buffer: row r (0..15) of a segment at r * kLmTRow; this lane writes row
  // 8 rg + lane / 8 at byte 16 (lane % 8) and reads, for step half hh, row lr at byte
  // 64 hh + 16 kg.
  unsigned char* tw0 = tb + lrow * kLmTRow + lbyte;
  unsigned char* tw1 = tw0 + 8 * kLmTRow;
  const unsigned char* trd = tb + lr * kLmTRow + 16 * kg;
  lds_barrier();  // vals initialised
  // One tile through this wave's slice: R holds its loads; with kNext they are replaced by
  // the next tile's (p0, p1) as they are consumed (the last tile loads nothing more).
  auto pass = [&](auto next_tag, const unsigned char* p0, const unsigned char* p1) {
    constexpr bool kNext = decltype(next_tag)::value;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < kSeg; ++c) {
      *reinterpret_cast<u32x4*>(tw0) = R[2 * c];
      *reinterpret_cast<u32x4*>(tw1) = R[2 * c + 1];
      if (kNext) {
        R[2 * c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p0 + 128 * c));
        R[2 * c + 1] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p1 + 128 * c));
      }
      const u32x4 b0 = *reinterpret_cast<const u32x4*>(trd);
      const u32x4 b1 = *reinterpret_cast<const u32x4*>(trd + 64);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(A[2 * c]), as_bf16x8(b0), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(A[2 * c + 1]), as_bf16x8(b1), acc, 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    return acc;
  };
  for (int j = 0; j < ntw; ++j) {
    const f32x4 acc = j + 1 < ntw ? pass(std::true_type{}, row_ptr(j + 1, 0), row_ptr(j + 1, 1))
                                  : pass(std::false_type{}, nullptr, nullptr);
    // This wave's partial: acc[jj] = sum over its slice for (row 4 kg + jj, column lr).
    float* rw = red + ((j & 1) * kLmWaves + w) * 256;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) rw[(4 * kg + jj) * 16 + lr] = acc[jj];
    lds_barrier();
    // Waves 0-3: one (row, column) each, the 8 partials summed in wave order.
    const int t = static_cast<int>(threadIdx.x);
    if (t < 256) {
      const float* rr = red + (j & 1) * kLmWaves * 256 + t;
      float sum = rr[0];
#pragma unroll
      for (int ww = 1; ww < kLmWaves; ++ww) sum += rr[ww * 256];
      const int row = t >> 4, col = t & 15;
      const int64_t v = static_cast<int64_t>(g + j * G) * 16 + col;
      if (row < Mg && v < a.V) vals[row * rstride + j * 16 + col] = sum;
    }
  }
  lds_barrier();
  // Slot s = 16 j + column holds vocabulary id 16 (g + j G) + column.
  emit_rows<NR>(a, vals, rstride, nslot, Mg, w, lane, (static_cast<int64_t>(grp) * G + g) * kLmRows,
                reinterpret_cast<uint64_t*>(tb), [&](int s2) { return static_cast<uint32_t>(static_cast<int64_t>(g + (s2 >> 4) * G) * 16 + (s2 & 15)); });
}

constexpr int kLmRankMax = 512;  // survivors ranked by counting; more take the radix selection

struct MergeLayout {
  uint32_t hist, misc, sel, surv, total;
};

__host__ __device__ inline MergeLayout merge_layout(int G, int K) {
  MergeLayout L{};
  L.hist = 0;                                     // uint32[256]
  L.misc = L.hist + 256 * 4;                      // uint32[4], float[4]
  L.sel = L.misc + 32;                            // uint64[K]
  L.surv = L.sel + static_cast<uint32_t>(K) * 8;  // uint64[G * K]
  L.total = L.surv + static_cast<uint32_t>(G) * K * 8;
  return L;
}

// Merge: one workgroup per row of h; wave 0 does the common case alone.
//  * LSE from the workgroups' (max, sum) pairs, each lane summing its workgroups in order.
//  * The K-th largest key kB among the lists' first two entries bounds the row's K-th:
//    at least K distinct entries have a key >= kB.  Every entry of the row's top K heads
//    its own sorted list down to keys >= kB, so the list prefixes with keys >= kB hold the
//    row's top K.  They are read in rounds (entry e of every list still above the bound)
//    and compacted to LDS.
//  * Up to kLmRankMax survivors are ranked by counting by all waves; more (most logits
//    tied) take an 8-bit radix selection of the K-th order value first.
// GL: lists per lane (G <= 64 GL).
template <int GL>
__global__ __launch_bounds__(kLmMergeThreads) void lm_head_merge_kernel(LmArgs a, int G) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int K = a.K;
  const MergeLayout L = merge_layout(G, K);
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem_raw + L.hist);
  uint32_t* misc = reinterpret_cast<uint32_t*>(smem_raw + L.misc);  // [0] count [1] need [2] digit
  float* mfl = reinterpret_cast<float*>(smem_raw + L.misc + 16);     // [0] max [1] log sum
  uint64_t* sel = reinterpret_cast<uint64_t*>(smem_raw + L.sel);
  uint64_t* surv = reinterpret_cast<uint64_t*>(smem_raw + L.surv);
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid % kWave;
  const int m = static_cast<int>(blockIdx.x);
  const int grp = m / kLmRows, mr = m % kLmRows;
  const int64_t base = static_cast<int64_t>(grp) * G * kLmRows + mr;  // workgroup g's partial: base + 16 g
  if (tid < kWave) {
    constexpr int R = 2 * GL;
    constexpr int kHead = 4;  // entries of every list read with the first loads
    float pm[GL], ps[GL];
    uint32_t key[R];
    const uint2* lst[GL];
    uint2 hd[GL][kHead];
#pragma unroll
    for (int i = 0; i < GL; ++i) {
      const int g = lane + kWave * i;
      const bool live = g < G;
      lst[i] = a.part_cand + (base + static_cast<int64_t>(live ? g : 0) * kLmRows) * K;
      const float2 p = live ? a.part_ms[base + static_cast<int64_t>(g) * kLmRows] : make_float2(neg_inf(), 0.f);
      pm[i] = p.x;
      ps[i] = p.y;
#pragma unroll
      for (int e = 0; e < kHead; ++e) hd[i][e] = live && e < K ? lst[i][e] : make_uint2(0u, 0u);
      key[2 * i] = hd[i][0].x;
      key[2 * i + 1] = hd[i][1].x;
    }
    float mx = neg_inf();
#pragma unroll
    for (int i = 0; i < GL; ++i) mx = fmaxf(mx, pm[i]);
    mx = wave_max(mx);
    float se = 0.f;
#pragma unroll
    for (int i = 0; i < GL; ++i)
      if (pm[i] != neg_inf()) se += ps[i] * __builtin_amdgcn_exp2f((pm[i] - mx) * kLog2e);
    se = wave_sum(se);
    const float lsum = __builtin_amdgcn_logf(se) * kLn2;
    // kB: the K-th largest nonzero top key (0, no pruning, when fewer than K).
    int n_nz = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) n_nz += popc(ballot(key[r] != 0u));
    uint32_t kb = 0u;
    if (n_nz >= K) {
      uint64_t sl[R];
      select_best<R>(key, n_nz, K, sl);
      uint32_t lo = ~0u;
#pragma unroll
      for (int r = 0; r < R; ++r) lo = min(lo, lane_in(sl[r]) ? key[r] : ~0u);
      kb = wave_umin(lo);
    }
    // Survivors: entry e of every list still above the bound, the first kHead entries
    // from the registers, later ones (rare) one round of loads each.
    int ns = 0;
    uint32_t open = 0u;  // bit i: list i still above the bound
#pragma unroll
    for (int i = 0; i < GL; ++i)
      if (lane + kWave * i < G) open |= 1u << i;
    auto take = [&](const uint2 (&c)[GL]) {
#pragma unroll
      for (int i = 0; i < GL; ++i) {
        const bool keep = ((open >> i) & 1u) && c[i].x != 0u && c[i].x >= kb;
        if (!keep) open &= ~(1u << i);
        const uint64_t mk = ballot(keep);
        if (keep) surv[ns + static_cast<int>(lanes_below(mk))] = lm_order(c[i].x, c[i].y);
        ns += popc(mk);
      }
    };
#pragma unroll
    for (int e = 0; e < kHead; ++e) {
      uint2 c[GL];
#pragma unroll
      for (int i = 0; i < GL; ++i) c[i] = hd[i][e];
      take(c);
    }
    for (int e = kHead; e < K; ++e) {
      if (ballot(open != 0u) == 0ull) break;
      uint2 c[GL];
#pragma unroll
      for (int i = 0; i < GL; ++i) c[i] = (open >> i) & 1u ? lst[i][e] : make_uint2(0u, 0u);
      take(c);
    }
    if (lane == 0) {
      misc[0] = static_cast<uint32_t>(ns);
      mfl[0] = mx;
      mfl[1] = lsum;
      if (a.lse) a.lse[m] = mx + lsum;
    }
  }
  __syncthreads();
  const int ns = static_cast<int>(misc[0]);
  const float mx = mfl[0], lsum = mfl[1];
  const int nk = ns < K ? ns : K;
  auto emit = [&](uint64_t me, int rank) {
    const float v = f32_key_value(static_cast<uint32_t>(me >> 32));
    const int64_t o = static_cast<int64_t>(m) * K + rank;
    a.cand_ids[o] = static_cast<int32_t>(~static_cast<uint32_t>(me));
    a.cand_logit[o] = v;
    // (u - max) - log sum exp(u - max): the error stays relative to the log-probability
    // itself when the logits are large.
    if (a.cand_logprob) a.cand_logprob[o] = (v - mx) - lsum;
  };
  if (ns <= kLmRankMax) {
    for (int i = tid; i < ns; i += kLmMergeThreads) {
      const uint64_t me = surv[i];
      int rank = 0;
      for (int j = 0; j < ns; ++j) rank += surv[j] > me ? 1 : 0;
      if (rank < K) emit(me, rank);
    }
    return;
  }
  // The nk-th largest order value (distinct values), 8 bits at a time from the top.
  int need = nk;
  uint64_t prefix = 0ull;
  for (int shift = 56; shift >= 0; shift -= 8) {
    hist[tid] = 0u;
    __syncthreads();
    const uint64_t hmask = shift == 56 ? 0ull : (~0ull << (shift + 8));
    for (int e = tid; e < ns; e += kLmMergeThreads) {
      const uint64_t v = surv[e];
      if (((v ^ prefix) & hmask) == 0ull) atomicAdd(&hist[(v >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < kWave) {
      // Lane l holds digits 4l .. 4l+3; entries with a larger digit: the suffix sum over
      // the lanes above, plus the larger digits of its own.
      const uint32_t c0 = hist[4 * lane], c1 = hist[4 * lane + 1], c2 = hist[4 * lane + 2], c3 = hist[4 * lane + 3];
      const uint32_t own = c0 + c1 + c2 + c3;
      uint32_t suf = own;  // sum over lanes >= l
      for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t y = __shfl_down(suf, off);
        if (lane + off < kWave) suf += y;
      }
      uint32_t above = suf - own;
      const uint32_t nd = static_cast<uint32_t>(need);
      if (above < nd && nd <= suf) {
        const uint32_t cs[4] = {c0, c1, c2, c3};
        for (int b = 3; b >= 0; --b) {
          if (above + cs[b] >= nd) {
            misc[2] = static_cast<uint32_t>(4 * lane + b);
            misc[1] = nd - above;
            break;
          }
          above += cs[b];
        }
      }
    }
    __syncthreads();
    prefix |= static_cast<uint64_t>(misc[2]) << shift;
    need = static_cast<int>(misc[1]);
    __syncthreads();
  }
  if (tid == 0) misc[0] = 0u;
  __syncthreads();
  for (int e = tid; e < ns; e += kLmMergeThreads)
    if (surv[e] >= prefix) sel[atomicAdd(&misc[0], 1u)] = surv[e];
  __syncthreads();
  for (int i = tid; i < nk; i += kLmMergeThreads) {
    const uint64_t me = sel[i];
    int rank = 0;
    for (int j = 0; j < nk; ++j) rank += sel[j] > me ? 1 : 0;
    emit(me, rank);
  }
}

int cu_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  return cus;
}

constexpr int kLmSplitMaxRounds = 96;  // tiles per workgroup of the split kernel (LDS: 16 x 96 x 16 logits)

// The split kernel runs when d = 256 * SW for an instantiated SW (whole 128-byte segments
// per wave slice, at most 2 x 20 operand registers of 4 dwords).
bool split_fits(int d) {
  if (d % 512 != 0) return false;
  const int sw = d / 256;
  return sw >= 4 && sw <= 20 && (sw <= 16 || sw == 20);
}

// Workgroups: one per compute unit, more if a workgroup's tiles would not fit its LDS,
// none without a tile.
int lm_grid(int n_tiles, int d) {
  const int cus = cu_count();
  if (split_fits(d)) {
    int G = cus;
    if ((n_tiles + kLmSplitMaxRounds - 1) / kLmSplitMaxRounds > G) G = (n_tiles + kLmSplitMaxRounds - 1) / kLmSplitMaxRounds;
    if (G > n_tiles) G = n_tiles;
    return G < 1 ? 1 : G;
  }
  const int per_wg = kLmWaves * kLmMaxRounds;
  int G = cus;
  if ((n_tiles + per_wg - 1) / per_wg > G) G = (n_tiles + per_wg - 1) / per_wg;
  const int useful = (n_tiles + kLmWaves - 1) / kLmWaves;
  if (G > useful) G = useful;
  return G < 1 ? 1 : G;
}

struct LmWorkspace {
  size_t ms, cand, total;
};

LmWorkspace lm_workspace(int M, int K, int G) {
  const size_t parts = static_cast<size_t>((M + kLmRows - 1) / kLmRows) * G * kLmRows;
  auto up = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  LmWorkspace w{};
  w.ms = 0;
  w.cand = up(parts * sizeof(float2));
  w.total = w.cand + up(parts * static_cast<size_t>(K) * sizeof(uint2));
  return w;
}

constexpr size_t kLmMaxLds = 160 * 1024;

}  // namespace

size_t lm_head_workspace_bytes(int M, int d, int64_t V, int K) {
  const int G = lm_grid(static_cast<int>((V + 15) / 16), d);
  if (G > 16 * kWave || merge_layout(G, K).total > kLmMaxLds) return 0;
  return lm_workspace(M, K, G).total;
}

hipError_t launch_lm_head_topk(const void* h, const void* w_lm, int M, int d, int64_t V, int K, int32_t* cand_ids,
                               float* cand_logit, float* cand_logprob, float* lse, void* workspace,
                               hipStream_t stream) {
  LmArgs a{};
  a.h = static_cast<const uint16_t*>(h);
  a.w = static_cast<const uint16_t*>(w_lm);
  a.M = M;
  a.d = d;
  a.K = K;
  a.V = V;
  a.n_tiles = static_cast<int>((V + 15) / 16);
  const int G = lm_grid(a.n_tiles, d);
  const bool split = split_fits(d);
  a.rounds = split ? (a.n_tiles + G - 1) / G : (a.n_tiles + G * kLmWaves - 1) / (G * kLmWaves);
  const LmWorkspace lw = lm_workspace(M, K, G);
  char* ws = static_cast<char*>(workspace);
  a.part_ms = reinterpret_cast<float2*>(ws + lw.ms);
  a.part_cand = reinterpret_cast<uint2*>(ws + lw.cand);
  a.cand_ids = cand_ids;
  a.cand_logit = cand_logit;
  a.cand_logprob = cand_logprob;
  a.lse = lse;
  const int groups = (M + kLmRows - 1) / kLmRows;
  const dim3 grid(static_cast<unsigned>(G), static_cast<unsigned>(groups)), block(kLmWaves * kWave);
  if (split) {
    const int rstride = a.rounds * 16 + kLmRowPad;
    const size_t smem = split_layout(rstride).total;
    const int nslot = a.rounds * 16;
    const int sw = d / 256;
#define UBT_LM_SPLIT(SWV, NRV)                                                                     \
  do {                                                                                             \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&lm_head_split_kernel<SWV, NRV>),     \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem)); \
    hipLaunchKernelGGL((lm_head_split_kernel<SWV, NRV>), grid, block, smem, stream, a);            \
  } while (0)
#define UBT_LM_SPLIT_NR(SWV)      \
  do {                            \
    if (nslot <= 4 * kWave)       \
      UBT_LM_SPLIT(SWV, 4);       \
    else if (nslot <= 10 * kWave) \
      UBT_LM_SPLIT(SWV, 10);      \
    else if (nslot <= 16 * kWave) \
      UBT_LM_SPLIT(SWV, 16);      \
    else                          \
      UBT_LM_SPLIT(SWV, 24);      \
  } while (0)
    switch (sw) {
      case 4: UBT_LM_SPLIT_NR(4); break;
      case 6: UBT_LM_SPLIT_NR(6); break;
      case 8: UBT_LM_SPLIT_NR(8); break;
      case 10: UBT_LM_SPLIT_NR(10); break;
      case 12: UBT_LM_SPLIT_NR(12); break;
      case 14: UBT_LM_SPLIT_NR(14); break;
      case 16: UBT_LM_SPLIT_NR(16); break;
      default: UBT_LM_SPLIT_NR(20); break;
    }
#undef UBT_LM_SPLIT_NR
#undef UBT_LM_SPLIT
  } else {
    const size_t smem = static_cast<size_t>(kLmRows) * (a.rounds * kLmWaves * 16 + kLmRowPad) * sizeof(float) +
                        kLmWaves * kLmStageWords * sizeof(uint64_t);  // + the per-wave stages
    const int nr = 2 * a.rounds;  // slots per lane: rounds * 128 / 64
    const bool p8 = (d / 32) % 8 == 0;
#define UBT_LM_LAUNCH(PP, NRV)                                                                     \
  do {                                                                                             \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&lm_head_stream_kernel<PP, NRV>),     \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem)); \
    hipLaunchKernelGGL((lm_head_stream_kernel<PP, NRV>), grid, block, smem, stream, a);            \
  } while (0)
#define UBT_LM_NR(PP)        \
  do {                       \
    if (nr <= 4)             \
      UBT_LM_LAUNCH(PP, 4);  \
    else if (nr <= 16)       \
      UBT_LM_LAUNCH(PP, 16); \
    else                     \
      UBT_LM_LAUNCH(PP, 32); \
  } while (0)
    if (p8)
      UBT_LM_NR(8);
    else
      UBT_LM_NR(1);
#undef UBT_LM_NR
#undef UBT_LM_LAUNCH
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t msmem = merge_layout(G, K).total;
  if (G <= 4 * kWave) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&lm_head_merge_kernel<4>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(msmem));
    hipLaunchKernelGGL((lm_head_merge_kernel<4>), dim3(static_cast<unsigned>(M)), dim3(kLmMergeThreads), msmem,
                       stream, a, G);
  } else {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&lm_head_merge_kernel<16>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(msmem));
    hipLaunchKernelGGL((lm_head_merge_kernel<16>), dim3(static_cast<unsigned>(M)), dim3(kLmMergeThreads), msmem,
                       stream, a, G);
  }
  return hipGetLastError();
}

}  // namespace ubt
