// Verification of a draft tree: tree attention, the acceptance walk and the KV commit.
//
// Appendix A / Verification via Tree-attention: the prefix-closed tree is verified in
// one target forward pass in which every node is evaluated under its own prefix (the
// committed context, then its ancestors and itself: the ancestor mask); the walk
// follows the child that matches the target's sample until the first mismatch, whose
// sample is the bonus token; the key/value rows along the accepted path are carried
// into the cache and the other branches are dropped.  Background, "Tree Drafting".
//
// Tree attention: one workgroup of 8 waves per (sequence, key/value head, group of up to
// 320 query rows).  The query rows of a key/value head are (node, head-in-group) pairs,
// node-major, so grouped heads share every key/value block, and the whole tree of a head
// fits one group at the usual shapes (65 nodes x 4 heads = 260 rows): keys and values are
// then read from HBM once.  Keys stream in blocks of 32 through LDS.  K is stored as it
// is; V is stored transposed (d-major), so both products read MFMA operands with plain
// LDS loads:
//   S^T = K Q^T     (v_mfma_f32_16x16x32_bf16, A = a K tile, B = 16 queries)
//   O^T += V^T P^T  (A = a V^T tile, B = P^T in the layout of the S^T accumulators)
// S^T puts the scores of one query in one lane column, 8 keys per lane, so P^T needs no
// shuffle: the k order of the second product is permuted to match (slot t of lane group
// g is key 4g + t for t < 4 and 16 + 4g + t - 4 after), and V^T is read in that order.
//
// The two products go to different waves.  Each SIMD holds a score wave (waves 0-3: the
// query fragments, S^T and the softmax) and an output wave (waves 4-7: the output
// accumulators and O^T), which share up to 5 query tiles of 16 rows.  The score wave
// hands the weights P^T of a block to its output wave through LDS, so while one wave runs
// the softmax on the vector ALU the other keeps the matrix core busy; each needs at most
// 256 registers.  The output wave runs one block behind.  A score wave computes the next
// block's scores tile by tile right after the tile's weights, so its own MFMAs overlap its
// vector work too.  K and V are staged through registers two steps ahead of their LDS
// stores, the output waves on even steps and the score waves on odd ones.  The running
// maximum is raised only when a score exceeds it by more than 2^8 (weights then stay
// below 256, exact enough in fp32 and bf16); it is checked on each block's scores as soon
// as they exist, and the factor by which the output must be rescaled goes to the output
// wave through LDS before that block's weights are used.
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kPairs = 4;                        // (score wave, output wave) pairs, one per SIMD
constexpr int kAttnWaves = 2 * kPairs;
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kStageThreads = kPairs * kWave;    // threads of one role, which stage K and V
constexpr int kMaxTiles = 5;                     // query tiles per pair
constexpr int kSlots = kPairs * kMaxTiles;       // query tiles per workgroup
constexpr int kAttnRows = 16 * kSlots;           // query rows per workgroup (320)
constexpr int kKB = 32;                          // keys per block
constexpr int kVtStride = 36;  // bf16 per V^T row: 32 keys + 4, so the transposing writes
                               // of one wave hit each bank at most twice
constexpr int kMaskWords = 8;  // mask words per node (N <= 256)
constexpr float kRescaleGap = 8.f;  // log2 units a score may exceed the running maximum

constexpr int kRing = 4;  // K and V blocks in LDS, loaded straight from global memory

template <int D>
struct AttnLds {
  uint16_t vt[3][D][kVtStride];       // V^T blocks i - 1 (read), i (transposed)
  v4u p[2][kSlots][kWave];            // P^T of blocks i (written) and i - 1 (read), per lane
  float alpha[3][kSlots][16];         // output rescale factor per query, blocks i - 1 .. i + 1
  uint32_t rescale[3][kPairs];        // nonzero: the pair's output must be rescaled first
  float fin_m[kSlots][16], fin_l[kSlots][16];  // final running maximum and sum per query
  uint32_t mask[kAttnRows][kMaskWords];         // the ancestor-mask rows of the group's nodes
};

typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));

__device__ __forceinline__ v8bf as_v8bf(v4u v) { return __builtin_bit_cast(v8bf, v); }

__device__ __forceinline__ v4f mfma_bf16(v4u a, v4u b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(a), as_v8bf(b), c, 0, 0, 0);
}

// Two floats to bf16, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((v2f{lo, hi}), v2bf));
}

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* prefix_len;
  const uint16_t* kt;
  const uint16_t* vt;
  const uint32_t* mask;
  const int32_t* n_nodes;
  int B, N, H, Hkv, g, R, groups;  // R = N * g query rows per key/value head, in groups of 320
  int64_t Pmax;
  float scale_log2;  // scale * log2(e)
  void* out;
  int out_f32;
  float* lse;
};

// Where the keys and values of block `blk` of sequence b, head h live: the context for
// blk < npb, else the tree.  Rows at or past `lim` do not exist; reads are clamped to row
// lim - 1.
struct BlockSrc {
  const uint16_t* k;
  const uint16_t* v;
  int64_t stride;  // rows of the source per sequence
  int base, lim;
};

__device__ __forceinline__ BlockSrc block_src(const AttnArgs& p, int blk, int npb, int P, int nn) {
  const bool tree = blk >= npb;
  return BlockSrc{tree ? p.kt : p.kc, tree ? p.vt : p.vc, tree ? static_cast<int64_t>(p.N) : p.Pmax,
                  tree ? (blk - npb) * kKB : blk * kKB, tree ? nn : P};
}

// K and V blocks go from global memory straight into LDS rings (global_load_lds, 16 bytes
// per lane, each wave instruction filling 1 KB of consecutive LDS), so the loads of
// several blocks are in flight without holding registers.  A block is 32 rows of D
// bf16, C = D / 8 chunks of 16 bytes per row; chunk c of row r sits at chunk position
// c ^ swz(r) of the row, which keeps the MFMA fragment reads (K) and the transposing
// reads (V) free of bank conflicts.  Rows past the block's end are copies of its last
// row: their weights are exactly 0 and their values finite.
__device__ __forceinline__ int swz_k(int row, int C) { return row & (C - 1); }
__device__ __forceinline__ int swz_v(int row, int C) { return (row >> 1) & (C - 1); }

// The loads of one block by one wave of a role (wave index wr, 0..3): C / 8 instructions.
// Lane offsets within a block (row r, chunk c) are fixed; `off` holds them in bytes for
// the wave's instructions.  The block's first row is a wave-uniform address; only a
// block shorter than 32 rows clamps each lane's row to its last.
template <int D, bool kV>
struct DmaLanes {
  static constexpr int C = D / 8;
  static constexpr int kRowsPer = kWave / C;  // rows per instruction
  static constexpr int kPerWave = C / 8;      // instructions per wave and block
  uint32_t off[kPerWave];
  int row[kPerWave];
  int wr;

  __device__ __forceinline__ DmaLanes(uint32_t row_bytes, int wave, int lane) : wr(wave) {
#pragma unroll
    for (int k = 0; k < kPerWave; ++k) {
      const int u = wr * kPerWave + k;
      const int r = u * kRowsPer + lane / C, pos = lane % C;
      const int c = pos ^ (kV ? swz_v(r, C) : swz_k(r, C));
      row[k] = r;
      off[k] = static_cast<uint32_t>(r) * row_bytes + 16u * static_cast<uint32_t>(c);
    }
  }

  __device__ __forceinline__ void load(const AttnArgs& p, const BlockSrc& bs, uint32_t row_bytes, uint16_t* slot,
                                       int b, int h) const {
    const char* first = reinterpret_cast<const char*>(kV ? bs.v : bs.k) +
                        (static_cast<int64_t>(b) * bs.stride + bs.base) * row_bytes + static_cast<int64_t>(h) * D * 2;
    const int rmax = bs.lim - 1 - bs.base;
    if (rmax >= kKB - 1) {
#pragma unroll
      for (int k = 0; k < kPerWave; ++k) {
        const void* src = first + off[k];
        __builtin_amdgcn_global_load_lds(src, slot + (wr * kPerWave + k) * kWave * 8, 16, 0, 0);
      }
    } else {
#pragma unroll
      for (int k = 0; k < kPerWave; ++k) {
        const void* src = first + (off[k] - static_cast<uint32_t>(row[k] - min(row[k], rmax)) * row_bytes);
        __builtin_amdgcn_global_load_lds(src, slot + (wr * kPerWave + k) * kWave * 8, 16, 0, 0);
      }
    }
  }
};

// V^T slot from a V ring slot: staging thread t (0 .. 255) takes keys 2 kp, 2 kp + 1 at
// the 8 d of chunk c and packs two keys per 32-bit LDS word.
template <int D>
__device__ __forceinline__ void transpose_v(AttnLds<D>& lds, int st, const uint16_t* vslot, int t) {
  constexpr int C = D / 8;
  const int kp = t % 16, c = t / 16;
  if (c < C) {
    const int r0 = 2 * kp;
    const int pos = c ^ swz_v(r0, C);  // the same for rows 2 kp and 2 kp + 1
    const v4u v0 = *reinterpret_cast<const v4u*>(vslot + r0 * D + 8 * pos);
    const v4u v1 = *reinterpret_cast<const v4u*>(vslot + (r0 + 1) * D + 8 * pos);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t a = (v0[e / 2] >> (16 * (e % 2))) & 0xFFFFu;
      const uint32_t bb = (v1[e / 2] >> (16 * (e % 2))) & 0xFFFFu;
      *reinterpret_cast<uint32_t*>(&lds.vt[st][8 * c + e][2 * kp]) = a | (bb << 16);
    }
  }
}

// A workgroup barrier after this wave's LDS writes and all but its N youngest loads have
// completed.  No release fence: such a fence would also wait for every load into LDS
// still in flight, which the rings keep several blocks deep.
template <int N>
__device__ __forceinline__ void ring_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));  // vmcnt(N), lgkmcnt(0)
  asm volatile("s_barrier" ::: "memory");
}

// The lane's 8 keys of a block as visibility bits: bit t is key 4 kg + t (t < 4) or
// 16 + 4 kg + t - 4 (t >= 4), the order of the score accumulators.
__device__ __forceinline__ uint32_t lane_bits(uint32_t keys32, int kg) {
  return ((keys32 >> (4 * kg)) & 0xFu) | (((keys32 >> (16 + 4 * kg)) & 0xFu) << 4);
}

// Which keys of a block a score wave's lane sees, per tile.  The context blocks come
// first, then the tree's; `ml` is the tile row's node in the mask rows staged in LDS, or
// -1 for a row with no query.
struct VisCtx {
  int P, npb, nn, kg;
};

template <int D>
__device__ __forceinline__ uint32_t tile_vis(const AttnLds<D>& lds, const VisCtx& v, int blk, int ml) {
  if (ml < 0) return 0u;
  if (blk < v.npb) {
    const int left = v.P - blk * kKB;  // >= 1 keys of the block inside the prefix
    return lane_bits(left >= kKB ? ~0u : ((1u << left) - 1u), v.kg);
  }
  const int tb = blk - v.npb;
  const int left = v.nn - tb * kKB;
  const uint32_t in = left >= kKB ? ~0u : ((1u << left) - 1u);
  return lane_bits(lds.mask[ml][tb] & in, v.kg);
}

// Largest visible score of a tile in log2 units (kAll: every key is visible).
template <bool kAll>
__device__ __forceinline__ float tile_max(v4f s0, v4f s1, uint32_t vis, float c) {
  float m;
  if (kAll) {
    m = fmaxf(fmaxf(fmaxf(s0[0], s0[1]), fmaxf(s0[2], s0[3])), fmaxf(fmaxf(s1[0], s1[1]), fmaxf(s1[2], s1[3])));
  } else {
    m = neg_inf();
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      m = ((vis >> e) & 1u) ? fmaxf(m, s0[e]) : m;
      m = ((vis >> (4 + e)) & 1u) ? fmaxf(m, s1[e]) : m;
    }
  }
  return m * c;
}

template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};

// Score wave state: query fragments, the score tiles of one block (keys 0..15 and
// 16..31), the running maximum (log2 units) and this lane's partial sum of weights.
template <int D, int TW>
struct ScoreState {
  v4u qf[TW][D / 32];
  v4f s0[TW], s1[TW];
  float m_run[TW], l_part[TW];
};

// The MFMA A fragment of K rows `row` (lane's row) at k step s from a ring slot.
template <int D>
__device__ __forceinline__ v4u k_frag(const uint16_t* kslot, int row, int s, int kg) {
  constexpr int C = D / 8;
  return *reinterpret_cast<const v4u*>(kslot + row * D + 8 * ((4 * s + kg) ^ swz_k(row, C)));
}

// The score tiles of the K ring slot `kslot` for every tile.
template <int D, int TW>
__device__ __forceinline__ void block_scores(const uint16_t* kslot, ScoreState<D, TW>& S, int lr, int kg) {
#pragma unroll
  for (int j = 0; j < TW; ++j) S.s0[j] = S.s1[j] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    const v4u a0 = k_frag<D>(kslot, lr, s, kg);
    const v4u a1 = k_frag<D>(kslot, 16 + lr, s, kg);
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      S.s0[j] = mfma_bf16(a0, S.qf[j][s], S.s0[j]);
      S.s1[j] = mfma_bf16(a1, S.qf[j][s], S.s1[j]);
    }
  }
}

// Raise the running maxima that fell more than the gap behind (uniform over each query's
// 4 lanes) and rescale the sums at once; the factors go to the output wave through LDS
// slot `as` with a flag, written for every block.
template <int D, int TW>
__device__ __forceinline__ void raise_max(AttnLds<D>& lds, int as, int pair, int lane, ScoreState<D, TW>& S,
                                          const float (&mx)[TW]) {
  bool grow = false;
#pragma unroll
  for (int j = 0; j < TW; ++j) grow = grow || (mx[j] > S.m_run[j] + kRescaleGap);
  const bool resc = ballot(grow) != 0ull;
  if (lane == 0) lds.rescale[as][pair] = resc ? 1u : 0u;
  if (resc) {
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      float m = mx[j];
      m = fmaxf(m, __shfl_xor(m, 16));
      m = fmaxf(m, __shfl_xor(m, 32));
      float alpha = 1.f;
      if (m > S.m_run[j] + kRescaleGap) {
        alpha = __builtin_amdgcn_exp2f(S.m_run[j] - m);
        S.m_run[j] = m;
        S.l_part[j] *= alpha;
      }
      if (lane < 16) lds.alpha[as][pair + kPairs * j][lane] = alpha;
    }
  }
}

// A score wave's step on block blk.  Tile by tile: the weights from the tile's scores,
// written to LDS for the output wave, then the next block's scores (K ring slot `kslot`)
// into the same registers, and the next block's maxima one tile behind.
// kFull: every key of the block is visible to every query; kFullNext: the same for the
// next block.
template <int D, int TW, bool kFull, bool kFullNext>
__device__ __forceinline__ void score_block(AttnLds<D>& lds, int blk, const uint16_t* kslot, int ps, int slot0,
                                            ScoreState<D, TW>& S, const VisCtx& vc, const int (&ml)[TW], float c,
                                            int lane, float (&mx_next)[TW]) {
  constexpr int DS = D / 32;
  const int lr = lane & 15, kg = lane >> 4;
  // The next block's maximum of tile j (none when this is the last block: its scores are
  // stale).
  const bool has_next = blk + 1 < vc.npb + (vc.nn + kKB - 1) / kKB;
  auto next_max = [&](int j) {
    const uint32_t vis = kFullNext ? 0xFFu : (has_next ? tile_vis<D>(lds, vc, blk + 1, ml[j]) : 0u);
    return tile_max<kFullNext>(S.s0[j], S.s1[j], vis, c);
  };
  v4u kf0[DS], kf1[DS];
#pragma unroll
  for (int s = 0; s < DS; ++s) {
    kf0[s] = k_frag<D>(kslot, lr, s, kg);
    kf1[s] = k_frag<D>(kslot, 16 + lr, s, kg);
  }
#pragma unroll
  for (int j = 0; j < TW; ++j) {
    // A stored row sees a visible key in its first block, so m_run is finite there.
    const float nm = -S.m_run[j];
    float pr[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      pr[e] = __builtin_amdgcn_exp2f(fmaf(S.s0[j][e], c, nm));
      pr[4 + e] = __builtin_amdgcn_exp2f(fmaf(S.s1[j][e], c, nm));
    }
    if (!kFull) {
      const uint32_t vis = tile_vis<D>(lds, vc, blk, ml[j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) pr[e] = ((vis >> e) & 1u) ? pr[e] : 0.f;
    }
    S.l_part[j] += ((pr[0] + pr[1]) + (pr[2] + pr[3])) + ((pr[4] + pr[5]) + (pr[6] + pr[7]));
    lds.p[ps][slot0 + kPairs * j][lane] = v4u{pack_bf16(pr[0], pr[1]), pack_bf16(pr[2], pr[3]),
                                              pack_bf16(pr[4], pr[5]), pack_bf16(pr[6], pr[7])};
    v4f n0 = v4f{0.f, 0.f, 0.f, 0.f}, n1 = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      n0 = mfma_bf16(kf0[s], S.qf[j][s], n0);
      n1 = mfma_bf16(kf1[s], S.qf[j][s], n1);
    }
    S.s0[j] = n0;
    S.s1[j] = n1;
    // The previous tile's next-block maximum, once its MFMAs have had this tile's vector
    // work to finish behind.
    if (j > 0) mx_next[j - 1] = next_max(j - 1);
  }
  mx_next[TW - 1] = next_max(TW - 1);
}

template <int D, int TW>
__global__ __launch_bounds__(kAttnThreads) void tree_attention_kernel(AttnArgs p) {
  constexpr int DS = D / 32;
  constexpr int DT = D / 16;
  constexpr int kBlkLoads = D / 64;  // loads per wave and block (C / 8)
  __shared__ AttnLds<D> lds;
  __shared__ __attribute__((aligned(16))) uint16_t k_ring[kRing][kKB * D];
  __shared__ __attribute__((aligned(16))) uint16_t v_ring[kRing][kKB * D];

  // Workgroup -> (sequence, key/value head, row group).  Consecutive workgroups go to
  // different XCDs; the remap puts the row groups of one (sequence, head) on one XCD, so
  // they share its key/value blocks through that XCD's L2.
  const int total = p.B * p.Hkv * p.groups;
  const int L = static_cast<int>(blockIdx.x);
  const int T8 = total - total % 8;
  const int id = L < T8 ? (L % 8) * (T8 / 8) + L / 8 : L;
  const int grp = id % p.groups;
  const int bh = id / p.groups;
  const int h = bh % p.Hkv;
  const int b = bh / p.Hkv;

  const int t = static_cast<int>(threadIdx.x);
  const int w = __builtin_amdgcn_readfirstlane(t / kWave);
  const int pair = w % kPairs;
  const bool scorer = w < kPairs;
  const int lane = t % kWave;
  const int lr = lane & 15, kg = lane >> 4;
  const int wr = w % kPairs;          // wave index within its role
  const int ts = t - kStageThreads;  // staging thread index of the output waves

  const int P = min(max(p.prefix_len[b], 0), static_cast<int>(p.Pmax));
  const int nn = min(max(p.n_nodes[b], 0), p.N);
  const int npb = (P + kKB - 1) / kKB;
  const int nblk = npb + (nn + kKB - 1) / kKB;
  const int words = (p.N + 31) / 32;

  // Tile j of this pair holds query rows r0 + 16 (pair + 4 j) + [0, 16) (slot pair + 4 j
  // of the LDS hand-over); this lane is the column lr of each.  Rows past R (and nodes
  // past n_nodes) have zero queries and are never stored.
  const int r0 = grp * kAttnRows;
  const int n_base = r0 / p.g;  // the group's first node
  // Row r of tile j: node r / g, head h g + r % g; a row has a query when r < R and its
  // node is below n_nodes.
  auto tile_row = [&](int j) { return r0 + 16 * (pair + kPairs * j) + lr; };
  auto has_query = [&](int r) { return r < p.R && r / p.g < nn; };
  const float c = p.scale_log2;

  // The mask rows of the group's nodes (at most 320) into LDS.
  const int n_hi = min(p.N, (r0 + kAttnRows + p.g - 1) / p.g);
  for (int e = t; e < (n_hi - n_base) * words; e += kAttnThreads) {
    const int ln = e / words, wd = e % words;
    lds.mask[ln][wd] = p.mask[(static_cast<int64_t>(b) * p.N + n_base + ln) * words + wd];
  }

  if (scorer) {
    // ---------------- score wave ----------------
    ScoreState<D, TW> S;
    int ml[TW];
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      const int r = tile_row(j);
      const bool live = has_query(r);
      ml[j] = live ? r / p.g - n_base : -1;
      const uint16_t* qr = p.q + ((static_cast<int64_t>(b) * p.N + (live ? r / p.g : 0)) * p.H + h * p.g +
                                  (live ? r % p.g : 0)) * D;
#pragma unroll
      for (int s = 0; s < DS; ++s) {
        const v4u v = *reinterpret_cast<const v4u*>(qr + 32 * s + 8 * kg);
        S.qf[j][s] = live ? v : v4u{0u, 0u, 0u, 0u};
      }
      S.l_part[j] = 0.f;
      S.m_run[j] = 0.f;
    }
    const VisCtx vc{P, npb, nn, kg};
    if (lane == 0) lds.rescale[0][pair] = 0u;
    // The score waves load V: block X goes to ring slot X % 4 at step X - 3 (blocks 0..2
    // before the first step); the output waves transpose it at step X.  Past the last
    // block the loads repeat it into free slots, so every step issues the same count.
    const int last = max(nblk - 1, 0);
    const uint32_t row_bytes = static_cast<uint32_t>(p.Hkv) * D * 2;
    const DmaLanes<D, true> dl(row_bytes, wr, lane);
    auto load_v_block = [&](int x) {
      dl.load(p, block_src(p, min(x, last), npb, P, nn), row_bytes, v_ring[x % kRing], b, h);
    };
    if (nblk > 0) {
      load_v_block(0);
      load_v_block(1);
      load_v_block(2);
    }
    ring_barrier<2 * kBlkLoads>();  // V block 0 and the mask rows are in; K blocks 0 and 1 too
    if (nblk > 0) {
      block_scores<D, TW>(k_ring[0], S, lr, kg);
      // A row with a query sees a key of its first block (key 0 of the context, or the
      // root), so its maximum is finite; rows with no query keep 0 and never rescale.
#pragma unroll
      for (int j = 0; j < TW; ++j) {
        float m = tile_max<false>(S.s0[j], S.s1[j], tile_vis<D>(lds, vc, 0, ml[j]), c);
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        S.m_run[j] = ml[j] >= 0 ? m : 0.f;
      }
    }
    ring_barrier<2 * kBlkLoads>();  // K slot 0 is refilled during the first step
    // One step per block; the last step's "next" scores come from a stale K slot and are
    // never used.  The rescale found on the next block's scores goes to the output wave
    // with it.  Before its barrier a step waits for V block blk + 1.
    auto step = [&](auto full, auto full_next, int blk) {
      if (nblk > 0) load_v_block(blk + 3);
      float mx[TW];
      score_block<D, TW, decltype(full)::value, decltype(full_next)::value>(lds, blk, k_ring[(blk + 1) % kRing],
                                                                           blk & 1, pair, S, vc, ml, c, lane, mx);
      raise_max<D, TW>(lds, (blk + 1) % 3, pair, lane, S, mx);
      ring_barrier<2 * kBlkLoads>();
    };
    // Blocks 0 .. nf - 1 lie wholly inside the context; each loop below runs one variant.
    const int nf = P / kKB;
    int blk = 0;
    for (; blk + 1 < nf; ++blk) step(BoolTag<true>{}, BoolTag<true>{}, blk);
    if (blk < nf) step(BoolTag<true>{}, BoolTag<false>{}, blk++);
    for (; blk < nblk; ++blk) step(BoolTag<false>{}, BoolTag<false>{}, blk);
    ring_barrier<0>();  // the output wave's last block; no load of this wave is left
    // Final maximum and sum per query for the output wave.
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      float l = S.l_part[j] + __shfl_xor(S.l_part[j], 16);
      l = l + __shfl_xor(l, 32);
      if (kg == 0) {
        lds.fin_m[pair + kPairs * j][lr] = S.m_run[j];
        lds.fin_l[pair + kPairs * j][lr] = l;
      }
    }
    ring_barrier<0>();
  } else {
    // ---------------- output wave ----------------
    v4f o[TW][DT];
#pragma unroll
    for (int j = 0; j < TW; ++j)
#pragma unroll
      for (int i = 0; i < DT; ++i) o[j][i] = v4f{0.f, 0.f, 0.f, 0.f};
    // The output waves load K: block X goes to ring slot X % 4 at step X - 4 (blocks 0..3
    // before the first step), and the score waves read it at step X - 1.  Past the last
    // block the loads repeat it into free slots, so every step issues the same count.
    const int last = max(nblk - 1, 0);
    const uint32_t row_bytes = static_cast<uint32_t>(p.Hkv) * D * 2;
    const DmaLanes<D, false> dl(row_bytes, wr, lane);
    auto load_k_block = [&](int x) {
      dl.load(p, block_src(p, min(x, last), npb, P, nn), row_bytes, k_ring[x % kRing], b, h);
    };
    if (nblk > 0) {
      load_k_block(0);
      load_k_block(1);
      load_k_block(2);
      load_k_block(3);
    }
    ring_barrier<2 * kBlkLoads>();  // K blocks 0 and 1 are in
    ring_barrier<2 * kBlkLoads>();  // the score waves have read K slot 0
    for (int blk = 0; blk <= nblk; ++blk) {
      if (nblk > 0) load_k_block(blk + 4);  // into the slot of block blk, read in the previous step
      // V^T of block blk (from its ring slot, in since the previous step's barrier) into
      // the slot of block blk - 3, read here three steps ago.
      if (blk < nblk) transpose_v<D>(lds, blk % 3, v_ring[blk % kRing], ts);
      if (blk > 0) {
        // O^T += V^T P^T for block blk - 1, after the rescale its scores asked for.
        const int qb = blk - 1, ps = qb & 1, vs = qb % 3;
        if (lds.rescale[vs][pair] != 0u) {
#pragma unroll
          for (int j = 0; j < TW; ++j) {
            const float a = lds.alpha[vs][pair + kPairs * j][lr];
#pragma unroll
            for (int i = 0; i < DT; ++i) o[j][i] *= a;
          }
        }
        v4u pt[TW];
#pragma unroll
        for (int j = 0; j < TW; ++j) pt[j] = lds.p[ps][pair + kPairs * j][lane];
#pragma unroll
        for (int i = 0; i < DT; ++i) {
          const uint16_t* vrow = &lds.vt[vs][16 * i + lr][0];
          const v2u lo = *reinterpret_cast<const v2u*>(vrow + 4 * kg);
          const v2u hi = *reinterpret_cast<const v2u*>(vrow + 16 + 4 * kg);
          const v4u a = v4u{lo.x, lo.y, hi.x, hi.y};
#pragma unroll
          for (int j = 0; j < TW; ++j) o[j][i] = mfma_bf16(a, pt[j], o[j][i]);
        }
      }
      ring_barrier<2 * kBlkLoads>();  // K block blk + 2 is in
    }
    ring_barrier<0>();  // the final statistics are in; no load of this wave is left
    // ---- normalise and store: lane (lr, kg) holds d = 16 i + 4 kg + e of its query ----
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      const int r = tile_row(j);
      if (r >= p.R) continue;
      const float l = lds.fin_l[pair + kPairs * j][lr];
      const bool has = has_query(r) && l > 0.f;
      const float inv = has ? 1.f / l : 0.f;
      const int64_t orow = (static_cast<int64_t>(b) * p.N + r / p.g) * p.H + h * p.g + r % p.g;
      if (p.out_f32) {
        float* op = static_cast<float*>(p.out) + orow * D;
#pragma unroll
        for (int i = 0; i < DT; ++i)
          *reinterpret_cast<v4f*>(op + 16 * i + 4 * kg) = has ? o[j][i] * inv : v4f{0.f, 0.f, 0.f, 0.f};
      } else {
        uint16_t* op = static_cast<uint16_t*>(p.out) + orow * D;
#pragma unroll
        for (int i = 0; i < DT; ++i) {
          const v4f v = has ? o[j][i] * inv : v4f{0.f, 0.f, 0.f, 0.f};
          *reinterpret_cast<v2u*>(op + 16 * i + 4 * kg) = v2u{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
        }
      }
      if (p.lse && kg == 0)
        p.lse[orow] = has ? (lds.fin_m[pair + kPairs * j][lr] + __builtin_amdgcn_logf(l)) * kLn2 : neg_inf();
    }
  }
}

// ---- acceptance walk: one wave per sequence ----------------------------------------------
__global__ __launch_bounds__(kWave) void verify_accept_kernel(const int32_t* __restrict__ token,
                                                              const int32_t* __restrict__ parent,
                                                              const int32_t* __restrict__ n_nodes,
                                                              const int32_t* __restrict__ target, int N,
                                                              int32_t* __restrict__ accept_len,
                                                              int32_t* __restrict__ accept_nodes,
                                                              int32_t* __restrict__ bonus) {
  const int b = static_cast<int>(blockIdx.x);
  const int lane = static_cast<int>(threadIdx.x);
  const int64_t o = static_cast<int64_t>(b) * N;
  const int nn = min(max(n_nodes[b], 1), N);
  int cur = 0, len = 0;
  // Each step moves to a larger node index (only nodes after `cur` are searched), so
  // the walk ends within N steps whatever the input.
  for (;;) {
    const int y = target[o + cur];
    int found = -1;
    for (int c0 = cur + 1; c0 < nn; c0 += kWave) {
      const int c = c0 + lane;
      const bool hit = c < nn && parent[o + c] == cur && token[o + c] == y;
      const uint64_t m = ballot(hit);
      if (m) {
        found = c0 + static_cast<int>(__builtin_ctzll(m));
        break;
      }
    }
    if (found < 0) {
      if (lane == 0) bonus[b] = y;
      break;
    }
    ++len;
    if (lane == 0) accept_nodes[o + len] = found;
    cur = found;
  }
  if (lane == 0) {
    accept_len[b] = len;
    accept_nodes[o] = 0;
  }
  for (int i = len + 1 + lane; i < N; i += kWave) accept_nodes[o + i] = -1;
}

// ---- KV commit: one workgroup per sequence ------------------------------------------------
__global__ __launch_bounds__(256) void commit_kv_kernel(const uint16_t* __restrict__ kt,
                                                        const uint16_t* __restrict__ vt,
                                                        const int32_t* __restrict__ accept_nodes,
                                                        const int32_t* __restrict__ accept_len, int32_t* prefix_len,
                                                        uint16_t* __restrict__ kc, uint16_t* __restrict__ vc, int N,
                                                        int rowv4, int64_t Pmax) {
  const int b = static_cast<int>(blockIdx.x);
  __shared__ int s_p, s_cnt;
  if (threadIdx.x == 0) {
    s_p = min(max(prefix_len[b], 0), static_cast<int>(Pmax));
    s_cnt = min(max(accept_len[b], 0), N - 1) + 1;
  }
  __syncthreads();
  const int P = s_p, cnt = s_cnt;
  const int64_t o = static_cast<int64_t>(b) * N;
  // rowv4 = 16-byte vectors per node row (H_kv * D * 2 / 16).
  for (int e = static_cast<int>(threadIdx.x); e < cnt * rowv4; e += static_cast<int>(blockDim.x)) {
    const int i = e / rowv4, c = e % rowv4;
    const int src = accept_nodes[o + i];
    if (P + i >= Pmax || src < 0 || src >= N) continue;
    const int64_t s = (o + src) * rowv4 + c;
    const int64_t d = (static_cast<int64_t>(b) * Pmax + P + i) * rowv4 + c;
    reinterpret_cast<v4u*>(kc)[d] = reinterpret_cast<const v4u*>(kt)[s];
    reinterpret_cast<v4u*>(vc)[d] = reinterpret_cast<const v4u*>(vt)[s];
  }
  __syncthreads();
  if (threadIdx.x == 0) prefix_len[b] = static_cast<int>(min(Pmax, static_cast<int64_t>(P) + cnt));
}

}  // namespace

hipError_t launch_tree_attention(const TreeAttnArgs& a, hipStream_t stream) {
  AttnArgs p{};
  p.q = static_cast<const uint16_t*>(a.q);
  p.kc = static_cast<const uint16_t*>(a.k_cache);
  p.vc = static_cast<const uint16_t*>(a.v_cache);
  p.prefix_len = a.prefix_len;
  p.kt = static_cast<const uint16_t*>(a.k_tree);
  p.vt = static_cast<const uint16_t*>(a.v_tree);
  p.mask = a.mask;
  p.n_nodes = a.n_nodes;
  p.B = a.B;
  p.N = a.N;
  p.H = a.H;
  p.Hkv = a.Hkv;
  p.g = a.H / a.Hkv;
  p.R = a.N * p.g;
  p.groups = (p.R + kAttnRows - 1) / kAttnRows;
  p.Pmax = a.Pmax;
  p.scale_log2 = a.scale * kLog2e;
  p.out = a.out;
  p.out_f32 = a.out_f32;
  p.lse = a.lse;
  const dim3 grid(static_cast<unsigned>(p.B * p.Hkv * p.groups));
  // Tiles per pair: enough for the group's rows (1, 3 or 5; rows past R are empty tiles).
  const int tiles = (min(p.R, kAttnRows) + 15) / 16;
  const int tw = (tiles + kPairs - 1) / kPairs;
  if (a.D == 128) {
    if (tw <= 1)
      hipLaunchKernelGGL((tree_attention_kernel<128, 1>), grid, dim3(kAttnThreads), 0, stream, p);
    else if (tw <= 3)
      hipLaunchKernelGGL((tree_attention_kernel<128, 3>), grid, dim3(kAttnThreads), 0, stream, p);
    else
      hipLaunchKernelGGL((tree_attention_kernel<128, kMaxTiles>), grid, dim3(kAttnThreads), 0, stream, p);
  } else {
    hipLaunchKernelGGL((tree_attention_kernel<64, kMaxTiles>), grid, dim3(kAttnThreads), 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_verify_accept(const int32_t* token, const int32_t* parent, const int32_t* n_nodes,
                                const int32_t* target, int B, int N, int32_t* accept_len, int32_t* accept_nodes,
                                int32_t* bonus, hipStream_t stream) {
  hipLaunchKernelGGL(verify_accept_kernel, dim3(static_cast<unsigned>(B)), dim3(kWave), 0, stream, token, parent,
                     n_nodes, target, N, accept_len, accept_nodes, bonus);
  return hipGetLastError();
}

hipError_t launch_commit_kv(const void* k_tree, const void* v_tree, const int32_t* accept_nodes,
                            const int32_t* accept_len, int32_t* prefix_len, void* k_cache, void* v_cache, int B, int N,
                            int Hkv, int D, int64_t Pmax, hipStream_t stream) {
  const int rowv4 = Hkv * D * 2 / 16;
  hipLaunchKernelGGL(commit_kv_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0, stream,
                     static_cast<const uint16_t*>(k_tree), static_cast<const uint16_t*>(v_tree), accept_nodes,
                     accept_len, prefix_len, static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), N,
                     rowv4, Pmax);
  return hipGetLastError();
}

}  // namespace ubt
