// Draft-tree construction from precomputed transition scores, and the ancestor mask.
//
// Appendix A, Algorithm 1: F_0 = {root}; for d = 1..gamma, E_d = F_{d-1} x C_d with
// l(y_{1:d}) = l(y_{1:d-1}) + log q_d^bi(y_d | y_{d-1}) + zeta (Eq. ubtree-depth-bonus),
// F_d = Top_W(E_d) (Eq. ubtree-frontier, W best extensions over all parents); then
// T = {root} + Top_budget(union of F_d) (Eq. ubtree-pruning).  Verification via
// Tree-attention: node n attends to itself and its ancestors -> packed mask rows.
//
// One wavefront per sequence; everything between the first load and the final stores
// lives in LDS and registers.  The score slabs of all depths are staged in LDS up front
// (when they fit).  Per depth the |F_{d-1}| * K extensions are scored in registers and
// Top_W is a ballot-driven radix selection on (score key, extension index); the W
// survivors are ranked among themselves to give F_d in order.  The same selection over
// the supertree gives the pruned tree, whose emission order is the ranking itself.
// Ties: score desc, then the extension index (parent position in F_{d-1}, then the
// candidate rank); across depths score desc, depth asc, position in F_d asc.
#include "bigram_tile.h"
#include "search.h"
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

constexpr int kMaxSlabFloats = 12288;  // 48 KB of staged score slabs
constexpr int kDraftWaves = 8;  // waves per workgroup of the one-launch selector + search

struct TreeSmem {
  float* slab;        // [gamma][K][K] when staged
  float* f_score;     // [gamma][W]
  uint32_t* f_info;   // [gamma][W]: parent position | candidate rank << 16
  int32_t* f_slot;    // [gamma][W]: output slot (-1 if not selected)
  uint32_t* s_key;    // [gamma][W]: key of the supertree entry (0 if empty)
  uint2* stage;       // [256] (key, sub) of staged entries
  float* stage_score; // [256] scores of staged frontier entries
  int32_t* par_slot;  // [256] parent slot of each emitted node
  int32_t* f_cnt;     // [gamma]
};

__host__ __device__ inline size_t tree_smem_bytes(int gamma, int K, int W, bool stage_slabs) {
  const size_t gw = static_cast<size_t>(gamma) * W;
  size_t bytes = 0;
  if (stage_slabs) bytes += static_cast<size_t>(gamma) * K * K * sizeof(float);
  bytes += gw * (sizeof(float) + sizeof(uint32_t) + sizeof(int32_t) + sizeof(uint32_t));
  bytes += kMaxNodes * (sizeof(uint2) + sizeof(float) + sizeof(int32_t));
  bytes += static_cast<size_t>(gamma) * sizeof(int32_t);
  return bytes;
}


// Ranks `n` staged (key, sub) entries by (key desc, sub asc) and calls emit(s, rank) for
// each entry s.
template <class Emit>
__device__ __forceinline__ void rank_staged(const uint2* stage, int n, int lane, Emit emit) {
  for (int s = lane; s < n; s += kWave) {
    const uint2 me = stage[s];
    int rank = 0;
    for (int t = 0; t < n; ++t) {
      const uint2 o = stage[t];
      rank += (o.x > me.x) || (o.x == me.x && o.y < me.y);
    }
    emit(s, rank);
  }
}

// Writes the selected entries (masks sel[]) of register rows into stage[0..); returns count.
template <int R>
__device__ __forceinline__ int stage_selected(uint2* stage, const uint32_t (&key)[R], const uint32_t (&sub)[R],
                                              const uint64_t (&sel)[R], int lane) {
  int n = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if ((sel[r] >> lane) & 1ull) stage[n + lanes_below(sel[r])] = make_uint2(key[r], sub[r]);
    n += popc(sel[r]);
  }
  __builtin_amdgcn_wave_barrier();
  return n;
}

template <int R>
__global__ __launch_bounds__(kWave) void build_tree_kernel(TreeArgs a, int stage_slabs, int vec_slabs,
                                                           uint64_t magic_k) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int lane = threadIdx.x;
  const int64_t b = blockIdx.x;
  const int gamma = a.gamma, K = a.K, W = a.W;
  const int GW = gamma * W;

  TreeSmem sm;
  {
    unsigned char* p = smem_raw;
    sm.slab = reinterpret_cast<float*>(p);
    if (stage_slabs) p += static_cast<size_t>(gamma) * K * K * sizeof(float);
    sm.f_score = reinterpret_cast<float*>(p);
    p += GW * sizeof(float);
    sm.f_info = reinterpret_cast<uint32_t*>(p);
    p += GW * sizeof(uint32_t);
    sm.f_slot = reinterpret_cast<int32_t*>(p);
    p += GW * sizeof(int32_t);
    sm.s_key = reinterpret_cast<uint32_t*>(p);
    p += GW * sizeof(uint32_t);
    sm.stage = reinterpret_cast<uint2*>(p);
    p += kMaxNodes * sizeof(uint2);
    sm.stage_score = reinterpret_cast<float*>(p);
    p += kMaxNodes * sizeof(float);
    sm.par_slot = reinterpret_cast<int32_t*>(p);
    p += kMaxNodes * sizeof(int32_t);
    sm.f_cnt = reinterpret_cast<int32_t*>(p);
  }

  const float* gslab = a.logq + b * gamma * K * K;
  if (stage_slabs) {
    const int n = gamma * K * K;  // a multiple of 4 floats when K is even
    if (vec_slabs) {
      const float4* src = reinterpret_cast<const float4*>(gslab);
      float4* dst = reinterpret_cast<float4*>(sm.slab);
      for (int e = lane; e < n / 4; e += kWave) dst[e] = src[e];
    } else {
      for (int e = lane; e < n; e += kWave) sm.slab[e] = gslab[e];
    }
  }
  for (int e = lane; e < GW; e += kWave) {
    sm.f_slot[e] = -1;
    sm.s_key[e] = 0;
  }
  __syncthreads();
  const float* slab = stage_slabs ? sm.slab : gslab;

  // ---- depth-wise expansion --------------------------------------------------------
  int np = 1;  // |F_{d-1}|
  for (int d = 1; d <= gamma; ++d) {
    const int n = np * K;
    const float* q = slab + static_cast<int64_t>(d - 1) * K * K;
    const float* prev_score = sm.f_score + (d > 1 ? (d - 2) * W : 0);
    const uint32_t* prev_info = sm.f_info + (d > 1 ? (d - 2) * W : 0);
    uint32_t key[R], sub[R];
    uint64_t live[R], sel[R];
    float sc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int e = r * kWave + lane;
      const bool ok = e < n;
      const int p = div_k(e, magic_k);
      const int c = e - p * K;
      float l = 0.f;
      if (ok) {
        const float base = d == 1 ? 0.f : prev_score[p];
        const int row = d == 1 ? 0 : static_cast<int>(prev_info[p] >> 16);
        l = (base + q[row * K + c]) + a.zeta;
      }
      sc[r] = l;
      key[r] = ok ? f32_key(l) : 0u;
      sub[r] = static_cast<uint32_t>(e);
      live[r] = ballot(ok);
    }
    const int w_d = n < W ? n : W;
    wave_select<R>(key, sub, live, w_d, 32, sel);
    // Stage the survivors with their scores.
    int cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if ((sel[r] >> lane) & 1ull) {
        const int pos = cnt + static_cast<int>(lanes_below(sel[r]));
        sm.stage[pos] = make_uint2(key[r], sub[r]);
        sm.stage_score[pos] = sc[r];
      }
      cnt += popc(sel[r]);
    }
    __builtin_amdgcn_wave_barrier();
    float* fs = sm.f_score + (d - 1) * W;
    uint32_t* fi = sm.f_info + (d - 1) * W;
    uint32_t* fk = sm.s_key + (d - 1) * W;
    rank_staged(sm.stage, cnt, lane, [&](int s, int rank) {
      const uint32_t e = sm.stage[s].y;
      const uint32_t p = static_cast<uint32_t>(div_k(static_cast<int>(e), magic_k));
      const uint32_t c = e - p * K;
      const float l = sm.stage_score[s];
      fs[rank] = l;
      fi[rank] = p | (c << 16);
      fk[rank] = sm.stage[s].x;
    });
    __builtin_amdgcn_wave_barrier();
    if (lane == 0) sm.f_cnt[d - 1] = cnt;
    if (a.f_count) {
      if (lane == 0) a.f_count[b * gamma + d - 1] = cnt;
      for (int j = lane; j < W; j += kWave) {
        const int64_t o = (b * gamma + d - 1) * W + j;
        const bool have = j < cnt;
        a.f_parent[o] = have ? static_cast<int32_t>(fi[j] & 0xFFFFu) : -1;
        a.f_cand[o] = have ? static_cast<int32_t>(fi[j] >> 16) : -1;
        a.f_score[o] = have ? fs[j] : neg_inf();
      }
    }
    __builtin_amdgcn_wave_barrier();
    np = cnt;
  }

  // ---- global pruning over the supertree --------------------------------------------
  // Entry f = (d-1)*W + j; order key (score key, (d-1) << 8 | j) -> desc, asc.
  int total = 0;
  for (int d = 0; d < gamma; ++d) total += sm.f_cnt[d];
  const int n_sel = total < a.budget ? total : a.budget;
  const int rows = (GW + kWave - 1) / kWave;
  uint32_t t = 0;
  {
    // Threshold on the score key: the n_sel-th largest.
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t cand = t | (1u << bit);
      int c = 0;
      for (int r = 0; r < rows; ++r) {
        const int f = r * kWave + lane;
        c += popc(ballot(f < GW && sm.s_key[f] >= cand));
      }
      if (c >= n_sel) t = cand;
    }
  }
  int above = 0, equal = 0;
  for (int r = 0; r < rows; ++r) {
    const int f = r * kWave + lane;
    const uint32_t k = f < GW ? sm.s_key[f] : 0u;
    above += popc(ballot(k > t));
    equal += popc(ballot(k == t && k != 0));
  }
  const int rest = n_sel - above;
  // Among entries tied at t, keep the `rest` with the smallest (depth, position).
  uint32_t t2 = 0xFFFFFFFFu;  // sub threshold: keep tied entries with sub <= t2
  if (rest > 0 && rest < equal) {
    uint32_t inv = 0;
    for (int bit = 15; bit >= 0; --bit) {
      const uint32_t cand = inv | (1u << bit);
      int c = 0;
      for (int r = 0; r < rows; ++r) {
        const int f = r * kWave + lane;
        const uint32_t k = f < GW ? sm.s_key[f] : 0u;
        const uint32_t subv = static_cast<uint32_t>(((f / W) << 8) | (f % W));
        c += popc(ballot(k == t && k != 0 && (0xFFFFu - subv) >= cand));
      }
      if (c >= rest) inv = cand;
    }
    t2 = 0xFFFFu - inv;
  }
  // Stage the selected supertree entries.
  int cnt = 0;
  for (int r = 0; r < rows; ++r) {
    const int f = r * kWave + lane;
    const uint32_t k = f < GW ? sm.s_key[f] : 0u;
    const uint32_t subv = f < GW ? static_cast<uint32_t>(((f / W) << 8) | (f % W)) : 0u;
    const bool take = k != 0 && (k > t || (k == t && rest > 0 && subv <= t2));
    const uint64_t m = ballot(take);
    if (take) sm.stage[cnt + lanes_below(m)] = make_uint2(k, subv);
    cnt += popc(m);
  }
  __builtin_amdgcn_wave_barrier();
  // cnt == n_sel.  Ranking gives the emission order; slot = 1 + rank.
  rank_staged(sm.stage, cnt, lane, [&](int s, int rank) {
    const uint32_t subv = sm.stage[s].y;
    const int f = static_cast<int>(subv >> 8) * W + static_cast<int>(subv & 0xFFu);
    sm.f_slot[f] = 1 + rank;
  });
  __syncthreads();

  const int N = a.budget + 1;
  const int words = (N + 31) / 32;
  const int n_nodes = 1 + cnt;
  int32_t* tok = a.token + b * N;
  int32_t* par = a.parent + b * N;
  int32_t* dep = a.depth + b * N;
  int32_t* crk = a.cand_rank + b * N;
  float* scr = a.score + b * N;
  if (lane == 0) {
    a.n_nodes[b] = n_nodes;
    tok[0] = a.anchor[b];
    par[0] = -1;
    dep[0] = 0;
    crk[0] = -1;
    scr[0] = 0.f;
    sm.par_slot[0] = -1;
  }
  for (int s = lane; s < cnt; s += kWave) {
    const uint32_t subv = sm.stage[s].y;
    const int d = static_cast<int>(subv >> 8) + 1;
    const int j = static_cast<int>(subv & 0xFFu);
    const int f = (d - 1) * W + j;
    const int slot = sm.f_slot[f];
    const uint32_t info = sm.f_info[f];
    const int p = static_cast<int>(info & 0xFFFFu);
    const int c = static_cast<int>(info >> 16);
    const int ps = d == 1 ? 0 : sm.f_slot[(d - 2) * W + p];
    tok[slot] = a.cand_ids[(b * gamma + d - 1) * K + c];
    par[slot] = ps;
    dep[slot] = d;
    crk[slot] = c;
    scr[slot] = sm.f_score[f];
    sm.par_slot[slot] = ps;
  }
  for (int n = n_nodes + lane; n < N; n += kWave) {
    tok[n] = -1;
    par[n] = -1;
    dep[n] = -1;
    crk[n] = -1;
    scr[n] = neg_inf();
  }
  __syncthreads();

  // ---- ancestor mask ------------------------------------------------------------------
  if (a.mask) {
    uint32_t* mrow = a.mask + b * static_cast<int64_t>(N) * words;
    for (int n = lane; n < N; n += kWave) {
      uint32_t wv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      if (n < n_nodes) {
        int m = n;
        for (int step = 0; step <= gamma && m >= 0; ++step) {
          const uint32_t bit = 1u << (m & 31);
          const int wi = m >> 5;
#pragma unroll
          for (int w = 0; w < 8; ++w) wv[w] |= (w == wi) ? bit : 0u;
          m = sm.par_slot[m];
        }
      }
#pragma unroll
      for (int w = 0; w < 8; ++w)
        if (w < words) mrow[n * words + w] = wv[w];
    }
  }
}


template <int KT, int R>
__global__ __launch_bounds__(kWave) void build_tree_fast_kernel(TreeArgs a, uint64_t magic_w) {
  static_assert(KT <= 16, "K = 64 runs build_tree_k64_kernel");
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int lane = threadIdx.x;
  const int64_t b = blockIdx.x;
  const int gamma = a.gamma;
  const FastSmem sm = fast_smem(smem_raw, fast_layout(gamma, KT, a.W));
  // Stage this sequence's score slabs and candidate ids.
  {
    const int ns = gamma * KT * KT;
    const float* gslab = a.logq + b * ns;
    if ((reinterpret_cast<uintptr_t>(gslab) & 15u) == 0) {
      const float4* src = reinterpret_cast<const float4*>(gslab);
      float4* dst = reinterpret_cast<float4*>(sm.slab);
#pragma unroll 4
      for (int e = lane; e < ns / 4; e += kWave) dst[e] = src[e];
    } else {
#pragma unroll 4
      for (int e = lane; e < ns; e += kWave) sm.slab[e] = gslab[e];
    }
  }
  const int32_t* gids = a.cand_ids + b * gamma * KT;
  for (int e = lane; e < gamma * KT; e += kWave) sm.cids[e] = gids[e];
  __syncthreads();
  slab_row_max<KT>(sm.slab, sm.rmax, lane, gamma * KT, kWave);
  __syncthreads();
  fast_search<KT, R, false>(a, sm, b, lane, magic_w);
}

// K = 64: kK64Waves waves search one sequence together, staging its slabs two depths at a
// time; wave 0 then prunes, emits the tree and builds the mask.  RW = registers of
// 64 entries per wave (W <= 4 RW).
template <int RW>
__global__ __launch_bounds__(kK64Waves* kWave) void build_tree_k64_kernel(TreeArgs a, uint64_t magic_w) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int64_t b = blockIdx.x;
  const int gamma = a.gamma;
  const FastSmem sm = fast_smem(smem_raw, fast_layout(gamma, 64, a.W));
  const int32_t* gids = a.cand_ids + b * gamma * 64;
  for (int e = static_cast<int>(threadIdx.x); e < gamma * 64; e += static_cast<int>(blockDim.x)) sm.cids[e] = gids[e];
  // (the first barrier of the expansion publishes the ids)
  int total = 0;
  if ((reinterpret_cast<uintptr_t>(a.logq) & 15u) == 0)
    expand_depths64<RW, true>(a, sm, b, w, lane, total);
  else
    expand_depths64<RW, false>(a, sm, b, w, lane, total);
  if (w != 0) return;
  finish_tree<64, false>(a, sm, b, lane, magic_w, total);
}

// K = 64: selector scores and tree search in one launch (the one-call draft step).
// Workgroups 0..B-1 search, one per sequence, as build_tree_k64_kernel does.  The other
// workgroups compute score slab t (position t / B of sequence t % B, depth-major, so the
// first positions' slabs come first) on four waves (bigram_split_tile), write it with
// agent-scope stores, wait until they have completed and set the slab's ready word.  A
// search wave waits for a slab's ready word before loading it, two depths ahead, so the
// search starts once its first two slabs exist and overlaps the rest of the selector.
// Slab workgroups never wait; a search wait that runs out of time marks its sequence
// with n_nodes = 0 and sets the error word.  The searcher clears the ready words of its
// sequence at the end (gamma <= 64, one lane each), so the next call starts from zero.
//
// The slab workgroups are persistent: slab_wgs of them take the slabs t, t + slab_wgs, ...
// in depth-major order.  One four-wave slab takes about 7 us from dispatch to its ready
// word even on an idle device (ids 0.4, row gathers 2.2, the hi/lo split and MFMAs 1.3,
// the LDS reduction 0.6, the epilogue and its stores 1.4 us), so the search starts about
// 7 us in however many run at once.  Measured at B = 32, gamma = 15, W = 12, r = 256 (us
// per step with the sweep): 32 slab workgroups 141.7, 64 97.9, 128 79.0, 256 78.7, one
// per slab (480) 79.4.
constexpr int kK64SlabRound = 8;  // slab workgroups per sequence

template <int RW>
__global__ __launch_bounds__(kK64Waves* kWave) __attribute__((amdgpu_waves_per_eu(2))) void draft_tree_k64_kernel(
    TreeArgs a, SelectorArgs s, uint32_t* ready, int slab_wgs, uint64_t magic_w) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int gamma = a.gamma;
  if (static_cast<int>(blockIdx.x) < a.B) {
    const int64_t b = blockIdx.x;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    const FastSmem sm = fast_smem(smem_raw, fast_layout(gamma, 64, a.W));
    const int32_t* gids = a.cand_ids + b * gamma * 64;
    for (int e = static_cast<int>(threadIdx.x); e < gamma * 64; e += static_cast<int>(blockDim.x))
      sm.cids[e] = gids[e];
    if (threadIdx.x == 0) *sm.fail = 0u;
    __syncthreads();
    int total = 0;
    expand_depths64<RW, false, true>(a, sm, b, w, lane, total, ready + b * gamma, t0);
    // Every wave has passed every wait (each depth ends with a workgroup barrier).
    if (w == 0 && lane < gamma) agent_store_u32(ready + b * gamma + lane, 0u);
    if (w != 0) return;
    finish_tree<64, true>(a, sm, b, lane, magic_w, total);
    return;
  }
  for (int t = static_cast<int>(blockIdx.x) - a.B; t < a.B * gamma; t += slab_wgs) {
    const int i = t / a.B;
    const int64_t b = t - i * a.B;
    const int64_t bi = b * gamma + i;
    bigram_split_tile<4, true, true>(s.phi, s.psi, s.gate + bi * s.r, s.V, s.r, i, 64, a.anchor + b,
                                     i > 0 ? a.cand_ids + (bi - 1) * 64 : a.cand_ids, a.cand_ids + bi * 64,
                                     s.cand_logit + bi * 64, s.sc.alpha[i], s.sc.lambda[i], nullptr,
                                     s.logq + bi * 64 * 64, reinterpret_cast<f32x4*>(smem_raw), w, lane);
    // Each wave's slab stores have completed before the workgroup barrier (which also
    // ends this slab's reads of the partial tiles); then the word.
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __syncthreads();
    if (threadIdx.x == 0) agent_store_u32(ready + bi, 1u);
  }
}

// Selector scores and tree search in one launch, one workgroup per sequence.  Wave 0
// computes the score slab of position 0 and starts searching; the other waves compute
// positions 1, 2, ... (round-robin) and publish each slab as it lands in LDS, and the
// search waits for a slab only when it first needs it.  Every slab also goes to global
// memory (logq).
template <int KT, int R>
__global__ __launch_bounds__(kDraftWaves* kWave) void draft_tree_fast_kernel(TreeArgs a, SelectorArgs s,
                                                                             uint64_t magic_w) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int nw = static_cast<int>(blockDim.x) / kWave;  // >= 2 when gamma >= 2
  const int64_t b = blockIdx.x;
  const int gamma = a.gamma;
  const FastSmem sm = fast_smem(smem_raw, fast_layout(gamma, KT, a.W));
  const int32_t* gids = a.cand_ids + b * gamma * KT;
  for (int e = static_cast<int>(threadIdx.x); e < gamma * KT; e += static_cast<int>(blockDim.x)) sm.cids[e] = gids[e];
  for (int e = static_cast<int>(threadIdx.x); e < gamma; e += static_cast<int>(blockDim.x)) sm.ready[e] = 0u;
  if (threadIdx.x == 0) *sm.fail = 0u;
  __syncthreads();
  const int first = w;
  const int stride = w == 0 ? gamma : nw - 1;
  for (int i = first; i < gamma; i += stride) {
    const int64_t bi = b * gamma + i;
    float* slab = sm.slab + i * KT * KT;
    bigram_tile_bf16<1>(s.phi, s.psi, s.gate + bi * s.r, s.V, s.r, i, KT, a.anchor + b,
                        i > 0 ? sm.cids + (i - 1) * KT : sm.cids, sm.cids + i * KT, s.cand_logit + bi * KT,
                        s.sc.alpha[i], s.sc.lambda[i], nullptr, slab, nullptr, lane);
    slab_row_max<KT>(sm.slab, sm.rmax, i * KT + lane, lane < KT ? i * KT + KT : 0, kWave);
    publish_slab(sm.ready, i);
    float* g = s.logq + bi * KT * KT;
#pragma unroll
    for (int e = lane; e < KT * KT; e += kWave) g[e] = slab[e];
  }
  if (w != 0) return;
  fast_search<KT, R, true>(a, sm, b, lane, magic_w);
}

__global__ __launch_bounds__(256) void tree_mask_kernel(const int32_t* __restrict__ parent,
                                                        const int32_t* __restrict__ n_nodes, int N,
                                                        uint32_t* __restrict__ mask) {
  __shared__ int32_t s_par[kMaxNodes];
  const int64_t b = blockIdx.x;
  const int words = (N + 31) / 32;
  int nn = n_nodes[b];
  nn = nn < 0 ? 0 : (nn > N ? N : nn);
  for (int n = threadIdx.x; n < N; n += blockDim.x) s_par[n] = parent[b * N + n];
  __syncthreads();
  uint32_t* mrow = mask + b * static_cast<int64_t>(N) * words;
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    uint32_t wv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (n < nn) {
      int m = n;
      // Walk towards the root; a pointer that does not decrease ends the walk.
      for (int step = 0; step < N; ++step) {
        const uint32_t bit = 1u << (m & 31);
        const int wi = m >> 5;
#pragma unroll
        for (int w = 0; w < 8; ++w) wv[w] |= (w == wi) ? bit : 0u;
        if (m == 0) break;
        const int p = s_par[m];
        if (p < 0 || p >= m) break;
        m = p;
      }
    }
#pragma unroll
    for (int w = 0; w < 8; ++w)
      if (w < words) mrow[n * words + w] = wv[w];
  }
}

}  // namespace

hipError_t launch_build_tree(const TreeArgs& a, hipStream_t stream) {
  const uint64_t magic_k = (0x100000000ull + a.K - 1) / a.K;  // ceil(2^32 / K)
  const dim3 grid(static_cast<unsigned>(a.B)), block(kWave);
  if (fast_tree_fits(a.gamma, a.K, a.W)) {
    const uint64_t magic_w = (0x100000000ull + a.W - 1) / a.W;
    const size_t smem = fast_layout(a.gamma, a.K, a.W).total;
    const int wk = a.W * a.K;
#define UBT_FAST_LAUNCH(KK, RR)                                                                              \
  do {                                                                                                       \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&build_tree_fast_kernel<KK, RR>),                \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));           \
    hipLaunchKernelGGL((build_tree_fast_kernel<KK, RR>), grid, block, smem, stream, a, magic_w);              \
  } while (0)
#define UBT_FAST_ROWS(KK)       \
  do {                          \
    if (wk <= 64)               \
      UBT_FAST_LAUNCH(KK, 1);   \
    else if (wk <= 128)         \
      UBT_FAST_LAUNCH(KK, 2);   \
    else if (wk <= 256)         \
      UBT_FAST_LAUNCH(KK, 4);   \
    else if (wk <= 384)         \
      UBT_FAST_LAUNCH(KK, 6);   \
    else                        \
      UBT_FAST_LAUNCH(KK, 8);   \
  } while (0)
#define UBT_K64_LAUNCH(RW)                                                                                   \
  do {                                                                                                       \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&build_tree_k64_kernel<RW>),                     \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));           \
    hipLaunchKernelGGL((build_tree_k64_kernel<RW>), grid, dim3(kK64Waves * kWave), smem, stream, a, magic_w); \
  } while (0)
    if (a.K == 4) {
      UBT_FAST_ROWS(4);
    } else if (a.K == 8) {
      UBT_FAST_ROWS(8);
    } else if (a.K == 16) {
      UBT_FAST_ROWS(16);
    } else if (a.W <= 4) {
      UBT_K64_LAUNCH(1);
    } else if (a.W <= 8) {
      UBT_K64_LAUNCH(2);
    } else if (a.W <= 12) {
      UBT_K64_LAUNCH(3);
    } else {
      UBT_K64_LAUNCH(4);
    }
#undef UBT_K64_LAUNCH
#undef UBT_FAST_ROWS
#undef UBT_FAST_LAUNCH
    return hipGetLastError();
  }
  const bool stage_slabs = static_cast<int64_t>(a.gamma) * a.K * a.K <= kMaxSlabFloats;
  const size_t smem = tree_smem_bytes(a.gamma, a.K, a.W, stage_slabs);
  const bool vec_slabs = (a.K % 2 == 0) && (reinterpret_cast<uintptr_t>(a.logq) % 16 == 0);
  const int n_max = a.W * a.K;
#define UBT_TREE_LAUNCH(RR)                                                                                \
  do {                                                                                                     \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&build_tree_kernel<RR>),                       \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));         \
    hipLaunchKernelGGL((build_tree_kernel<RR>), grid, block, smem, stream, a, stage_slabs ? 1 : 0,           \
                       vec_slabs ? 1 : 0, magic_k);                                                        \
  } while (0)
  if (n_max <= 64)
    UBT_TREE_LAUNCH(1);
  else if (n_max <= 128)
    UBT_TREE_LAUNCH(2);
  else if (n_max <= 256)
    UBT_TREE_LAUNCH(4);
  else if (n_max <= 512)
    UBT_TREE_LAUNCH(8);
  else if (n_max <= 1024)
    UBT_TREE_LAUNCH(16);
  else if (n_max <= 2048)
    UBT_TREE_LAUNCH(32);
  else
    UBT_TREE_LAUNCH(64);
#undef UBT_TREE_LAUNCH
  return hipGetLastError();
}

bool draft_tree_fused(int feat_dtype, int gamma, int K, int W) {
  return feat_dtype == 1 && K <= 16 && fast_tree_fits(gamma, K, W);
}

hipError_t launch_draft_tree(const SelectorArgs& s, const TreeArgs& a, hipStream_t stream) {
  const uint64_t magic_w = (0x100000000ull + a.W - 1) / a.W;
  const size_t smem = fast_layout(a.gamma, a.K, a.W).total;
  const int wk = a.W * a.K;
  const int nw = a.gamma < kDraftWaves ? a.gamma : kDraftWaves;
  const dim3 grid(static_cast<unsigned>(a.B)), block(static_cast<unsigned>(nw * kWave));
#define UBT_DRAFT_LAUNCH(KK, RR)                                                                             \
  do {                                                                                                       \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&draft_tree_fast_kernel<KK, RR>),                \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));           \
    hipLaunchKernelGGL((draft_tree_fast_kernel<KK, RR>), grid, block, smem, stream, a, s, magic_w);           \
  } while (0)
#define UBT_DRAFT_ROWS(KK)      \
  do {                          \
    if (wk <= 64)               \
      UBT_DRAFT_LAUNCH(KK, 1);  \
    else if (wk <= 128)         \
      UBT_DRAFT_LAUNCH(KK, 2);  \
    else if (wk <= 256)         \
      UBT_DRAFT_LAUNCH(KK, 4);  \
    else if (wk <= 384)         \
      UBT_DRAFT_LAUNCH(KK, 6);  \
    else                        \
      UBT_DRAFT_LAUNCH(KK, 8);  \
  } while (0)
  if (a.K == 4)
    UBT_DRAFT_ROWS(4);
  else if (a.K == 8)
    UBT_DRAFT_ROWS(8);
  else
    UBT_DRAFT_ROWS(16);
#undef UBT_DRAFT_ROWS
#undef UBT_DRAFT_LAUNCH
  return hipGetLastError();
}

bool draft_tree_k64_fused(int feat_dtype, int gamma, int K, int W) {
  return feat_dtype == 1 && K == 64 && fast_tree_fits(gamma, K, W);
}

hipError_t launch_draft_tree_k64(const SelectorArgs& s, const TreeArgs& a, uint32_t* ready, hipStream_t stream) {
  const uint64_t magic_w = (0x100000000ull + a.W - 1) / a.W;
  const size_t search_smem = fast_layout(a.gamma, 64, a.W).total;
  const size_t slab_smem = kSplitPartBytes<4>;
  const size_t smem = search_smem > slab_smem ? search_smem : slab_smem;
  const int slabs = a.B * a.gamma;
  const int slab_wgs = slabs < kK64SlabRound * a.B ? slabs : kK64SlabRound * a.B;
  const dim3 grid(static_cast<unsigned>(a.B + slab_wgs)), block(kK64Waves * kWave);
#define UBT_K64_DRAFT(RW)                                                                                    \
  do {                                                                                                       \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&draft_tree_k64_kernel<RW>),                     \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));           \
    hipLaunchKernelGGL((draft_tree_k64_kernel<RW>), grid, block, smem, stream, a, s, ready, slab_wgs, magic_w); \
  } while (0)
  if (a.W <= 4)
    UBT_K64_DRAFT(1);
  else if (a.W <= 8)
    UBT_K64_DRAFT(2);
  else if (a.W <= 12)
    UBT_K64_DRAFT(3);
  else
    UBT_K64_DRAFT(4);
#undef UBT_K64_DRAFT
  return hipGetLastError();
}

hipError_t launch_tree_mask(const int32_t* parent, const int32_t* n_nodes, int B, int N, uint32_t* mask,
                            hipStream_t stream) {
  hipLaunchKernelGGL(tree_mask_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0, stream, parent, n_nodes, N,
                     mask);
  return hipGetLastError();
}

}  // namespace ubt
