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
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

constexpr int kMaxSlabFloats = 12288;  // 48 KB of staged score slabs
constexpr int kMaxNodes = 256;
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

// e / K for 0 <= e < 2^16 and 1 <= K <= 64, with magic = ceil(2^32 / K).
__device__ __forceinline__ int div_k(int e, uint64_t magic) {
  return static_cast<int>((static_cast<uint64_t>(static_cast<uint32_t>(e)) * magic) >> 32);
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

// ---- register-resident search for the common shapes ---------------------------------
//
// Used when K is 4, 8 or 16, W <= 64, W*K <= 512 and gamma*W <= 1024.  Same results as
// the kernel above.  One wave runs alone per sequence, so a wave issues roughly one
// instruction per four cycles and every dependent LDS round trip is exposed: the layout
// is chosen to keep both counts low per depth.
//  * F_{d-1} is held one entry per lane (score key, position).  Each parent lane has its
//    slab row q_d[c_p][.] prefetched into registers and writes its K children to a
//    transpose buffer at index p*K + c, read back 64 entries per row.
//  * Top_W is a ballot radix selection over the bits below the common prefix of the live
//    keys (from a DPP max/min), stopping at the first bit that splits exactly W entries
//    off; a tie exactly at the boundary is resolved by index with mbcnt.
//  * the W survivors are compacted to LDS and each lane ranks its own entry against all
//    of them with broadcast reads, so F_d needs no sort and no reordering of registers.
//  * the supertree keys of all depths are loaded once into registers for Top_budget;
//    the ancestor mask is built by pointer jumping (ceil(log2(gamma+1)) rounds).
constexpr int kFastMaxWK = 512;
constexpr int kFastMaxGW = 1024;
constexpr int kFastMaxW = 64;
constexpr int kStageLive = 272;                // up to 255 selected entries + 16 zero entries
constexpr int kStageCap = kStageLive + kWave;  // + one dummy slot per lane
constexpr int kMaskWords = 8;                  // ceil(256 / 32)

struct FastLayout {
  uint32_t slab, rmax, cids, xpose, stage, s_key, s_info, f_slot, anc, mk, ready, total;
};

__host__ __device__ inline FastLayout fast_layout(int gamma, int K, int W) {
  FastLayout L{};
  uint32_t p = 0;
  auto take = [&p](size_t bytes) {
    const uint32_t at = p;
    p += static_cast<uint32_t>((bytes + 15) & ~static_cast<size_t>(15));
    return at;
  };
  L.slab = take(static_cast<size_t>(gamma) * K * K * sizeof(float));
  L.rmax = take(static_cast<size_t>(gamma) * K * sizeof(float));
  L.cids = take(static_cast<size_t>(gamma) * K * sizeof(int32_t));
  L.xpose = take(kFastMaxWK * sizeof(float));
  L.stage = take(kStageCap * sizeof(uint2));
  L.s_key = take(static_cast<size_t>(gamma) * W * sizeof(uint32_t));
  L.s_info = take(static_cast<size_t>(gamma) * W * sizeof(uint32_t));
  L.f_slot = take(static_cast<size_t>(gamma) * W * sizeof(int32_t));
  L.anc = take(kMaxNodes * sizeof(int32_t));
  L.mk = take(kMaxNodes * kMaskWords * sizeof(uint32_t));
  L.ready = take(static_cast<size_t>(gamma) * sizeof(uint32_t));
  L.total = p;
  return L;
}

__host__ __device__ inline bool fast_tree_fits(int gamma, int K, int W) {
  return (K == 4 || K == 8 || K == 16) && W <= kFastMaxW && W * K <= kFastMaxWK && gamma * W <= kFastMaxGW;
}

// Selects the `need` best live entries under (key desc, index asc), where entry (r, lane)
// has index r*64 + lane and key 0 marks a dead entry (rows past the data hold key 0).
// kmax and kmin, if given (kmin != 0), are the largest live key and a lower bound of the
// need-th largest one; otherwise they are taken from the keys.
template <int R>
__device__ __forceinline__ void select_best(const uint32_t (&key)[R], int n_live, int need, uint64_t (&sel)[R],
                                            uint32_t kmax = 0u, uint32_t kmin = 0u) {
  if (n_live <= need) {
#pragma unroll
    for (int r = 0; r < R; ++r) sel[r] = ballot(key[r] != 0u);
    return;
  }
  if (kmin == 0u) {
    uint32_t hi = 0, lo = ~0u;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      hi = max(hi, key[r]);
      lo = min(lo, key[r] != 0u ? key[r] : ~0u);
    }
    kmax = wave_umax(hi);
    kmin = wave_umin(lo);
  }
  // The need-th largest key lies in [kmin, kmax], so it shares the bits above the
  // highest bit where the two differ.
  uint32_t t = kmax;
  if (kmax != kmin) {
    uint32_t m = 0x80000000u >> __clz(kmax ^ kmin);
    t = kmax & ~(m | (m - 1u));
    // One exit: the loop ends at an exact split (the entries at or above cand) or after
    // the last bit, with t the need-th largest key.
    int cnt;
    do {
      const uint32_t cand = t | m;
      cnt = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        sel[r] = ballot(key[r] >= cand);
        cnt += popc(sel[r]);
      }
      t = cnt > need ? cand : t;
      m = radix_next(m, cnt, need, 0u);
    } while (m != 0u);
    if (cnt == need) return;
  }
  // t is the need-th largest key: take every key above t and the entries equal to t of
  // smallest index.
  int left = need;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    sel[r] = ballot(key[r] > t);
    left -= popc(sel[r]);
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint64_t eq = ballot(key[r] == t);
    const int c = popc(eq);
    if (left >= c) {
      sel[r] |= eq;
      left -= c;
    } else if (left > 0) {
      sel[r] |= ballot(lane_in(eq) && static_cast<int>(lanes_below(eq)) < left);
      left = 0;
    }
  }
}

// Writes the selected entries to stage[0..n) in index order as (x = ~index, y = key), so
// that the 64-bit value y:x orders entries by (key desc, index asc), then 16 zero
// entries.  Lanes with nothing to write store to their own dummy slot (no branches).
template <int R>
__device__ __forceinline__ void compact_selected(uint2* stage, const uint32_t (&key)[R], const uint64_t (&sel)[R],
                                                 int n, int lane) {
  const int dummy = kStageLive + lane;
  int pos = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int at = lane_in(sel[r]) ? pos + static_cast<int>(lanes_below(sel[r])) : dummy;
    stage[at] = make_uint2(~static_cast<uint32_t>(r * kWave + lane), key[r]);
    pos += popc(sel[r]);
  }
  stage[lane < 16 ? n + lane : dummy] = make_uint2(0u, 0u);
  __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ uint64_t order_value(uint32_t x, uint32_t y) {
  return (static_cast<uint64_t>(y) << 32) | x;
}

// Number of the n staged entries that come before `mine`.  Entries n..n+15 are zero, so
// whole chunks of 16 entries are compared; the next chunk is loaded before the current
// one is compared.
__device__ __forceinline__ int rank_in_stage(const uint2* stage, int n, uint64_t mine) {
  const uint4* s4 = reinterpret_cast<const uint4*>(stage);
  const int chunks = (n + 15) >> 4;
  uint4 cur[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) cur[i] = s4[i];
  int rank = 0;
  for (int ch = 0; ch < chunks; ++ch) {
    uint4 nxt[8];
    if (ch + 1 < chunks) {
#pragma unroll
      for (int i = 0; i < 8; ++i) nxt[i] = s4[(ch + 1) * 8 + i];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      rank += order_value(cur[i].x, cur[i].y) > mine ? 1 : 0;
      rank += order_value(cur[i].z, cur[i].w) > mine ? 1 : 0;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) cur[i] = nxt[i];
  }
  return rank;
}

template <int KT>
__device__ __forceinline__ void load_row(const float* row, float (&v)[KT]) {
#pragma unroll
  for (int i = 0; i < KT / 4; ++i) {
    const float4 t = reinterpret_cast<const float4*>(row)[i];
    v[4 * i] = t.x;
    v[4 * i + 1] = t.y;
    v[4 * i + 2] = t.z;
    v[4 * i + 3] = t.w;
  }
}

struct FastSmem {
  float* slab;
  float* rmax;  // per slab row: its largest entry
  int32_t* cids;
  float* xpose;
  uint2* stage;
  uint32_t* s_key;
  uint32_t* s_info;
  int32_t* f_slot;
  int32_t* anc;
  uint32_t* mk;
  uint32_t* ready;  // per position: its slab is in LDS (one-launch kernel only)
};

// Top_budget over the supertree: stages the selected entries (as compact_selected does).
template <int RS>
__device__ __forceinline__ void prune_supertree(const FastSmem& sm, int GW, int total, int n_sel, int lane) {
  uint32_t skey[RS];
#pragma unroll
  for (int r = 0; r < RS; ++r) {
    const int f = r * kWave + lane;
    const uint32_t k = sm.s_key[f < GW ? f : GW - 1];
    skey[r] = f < GW ? k : 0u;
  }
  uint64_t ssel[RS];
  select_best<RS>(skey, total, n_sel, ssel);
  compact_selected<RS>(sm.stage, skey, ssel, n_sel, lane);
}

__device__ __forceinline__ FastSmem fast_smem(unsigned char* raw, const FastLayout& L) {
  FastSmem sm;
  sm.slab = reinterpret_cast<float*>(raw + L.slab);
  sm.rmax = reinterpret_cast<float*>(raw + L.rmax);
  sm.cids = reinterpret_cast<int32_t*>(raw + L.cids);
  sm.xpose = reinterpret_cast<float*>(raw + L.xpose);
  sm.stage = reinterpret_cast<uint2*>(raw + L.stage);
  sm.s_key = reinterpret_cast<uint32_t*>(raw + L.s_key);
  sm.s_info = reinterpret_cast<uint32_t*>(raw + L.s_info);
  sm.f_slot = reinterpret_cast<int32_t*>(raw + L.f_slot);
  sm.anc = reinterpret_cast<int32_t*>(raw + L.anc);
  sm.mk = reinterpret_cast<uint32_t*>(raw + L.mk);
  sm.ready = reinterpret_cast<uint32_t*>(raw + L.ready);
  return sm;
}

// rmax[e] = the largest entry of slab row e, for rows e0, e0 + stride, ... < e1.
template <int KT>
__device__ __forceinline__ void slab_row_max(const float* slab, float* rmax, int e0, int e1, int stride) {
  for (int e = e0; e < e1; e += stride) {
    float v[KT];
    load_row<KT>(slab + e * KT, v);
    float m = v[0];
#pragma unroll
    for (int c = 1; c < KT; ++c) m = fmaxf(m, v[c]);
    rmax[e] = m;
  }
}

// Publishes slab i to the workgroup: every lane's earlier LDS writes complete before the
// flag is set.
__device__ __forceinline__ void publish_slab(uint32_t* ready, int i) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __hip_atomic_store(&ready[i], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Waits until slab i has been published.  Its producer is another wave of the same
// workgroup that runs unconditionally, so the flag is always set; the wait is bounded
// all the same.
__device__ __forceinline__ void wait_slab(uint32_t* ready, int i) {
  for (int spin = 0; spin < (1 << 22); ++spin) {
    const uint32_t f = __hip_atomic_load(&ready[i], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
    if (__builtin_amdgcn_readfirstlane(f) != 0u) return;
    __builtin_amdgcn_s_sleep(1);
  }
}

// Depth-wise expansion (Eq. ubtree-frontier): F_d = Top_W(E_d) for d = 1..gamma.  F_d is
// ranked (score desc, parent position, candidate rank) as it is formed and stored in that
// order to s_key / s_info (parent = its position in F_{d-1}), with the supertree outputs
// if asked.  total = the number of supertree nodes.
template <int KT, int R, bool kWait>
__device__ __forceinline__ void expand_depths(const TreeArgs& a, const FastSmem& sm, int64_t b, int lane,
                                              int& total) {
  constexpr int kLogK = KT == 4 ? 2 : (KT == 8 ? 3 : 4);
  const int gamma = a.gamma, W = a.W;
  // Frontier entry on lane j < np: score key, position in F, and its slab row for the
  // next depth (prefetched as soon as the entry's candidate rank is known).
  uint32_t fkey = f32_key(0.f);
  int fpos = 0;
  float nq[KT];
  if (kWait) wait_slab(sm.ready, 0);
  load_row<KT>(sm.slab, nq);  // depth 1 extends the root through row 0
  float rm = sm.rmax[0];
  int np = 1;
  total = 0;
  const float zeta = a.zeta;
  const bool with_zeta = zeta != 0.f;
  for (int d = 1; d <= gamma; ++d) {
    // Each parent's best child comes from its row maximum (rounding is monotone, so it
    // is exactly the largest of the children computed below).  With at least W parents,
    // W extensions reach the smallest of these, a lower bound of the W-th best one.
    uint32_t best_key = 0u;
    if (lane < np) {
      const float base = f32_key_value(fkey);
      float v[KT];
#pragma unroll
      for (int c = 0; c < KT; ++c) v[c] = base + nq[c];
      float best = base + rm;
      if (with_zeta) {
#pragma unroll
        for (int c = 0; c < KT; ++c) v[c] += zeta;
        best += zeta;
      }
      best_key = f32_key(best);
      float4* dst = reinterpret_cast<float4*>(sm.xpose + fpos * KT);
#pragma unroll
      for (int i = 0; i < KT / 4; ++i) dst[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
    }
    __builtin_amdgcn_wave_barrier();
    const int n = np * KT;
    uint32_t key[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int e = r * kWave + lane;
      const float x = sm.xpose[e];
      key[r] = e < n ? f32_key(x) : 0u;
    }
    const int w_d = n < W ? n : W;
    uint64_t sel[R];
    if (np >= W) {
      const uint32_t kmax = wave_umax(best_key);
      const uint32_t kbound = wave_umin(lane < np ? best_key : ~0u);
      select_best<R>(key, n, w_d, sel, kmax, kbound);
    } else {
      select_best<R>(key, n, w_d, sel);
    }
    compact_selected<R>(sm.stage, key, sel, w_d, lane);
    const uint2 st = sm.stage[lane];
    const bool have = lane < w_d;
    const uint32_t mx = have ? st.x : 0u, my = have ? st.y : 0u;
    const int e = have ? static_cast<int>(~mx) : 0;
    const int p = e >> kLogK;
    const int c = e & (KT - 1);
    if (d < gamma) {
      if (kWait) wait_slab(sm.ready, d);
      load_row<KT>(sm.slab + (d * KT + c) * KT, nq);
      rm = sm.rmax[d * KT + c];
    }
    const int rank = rank_in_stage(sm.stage, w_d, order_value(mx, my));
    const int fb = (d - 1) * W;
    if (have) {
      sm.s_key[fb + rank] = my;
      sm.s_info[fb + rank] = static_cast<uint32_t>(p) | (static_cast<uint32_t>(c) << 16);
    } else if (lane < W) {
      sm.s_key[fb + lane] = 0u;
    }
    if (a.f_count) {
      if (lane == 0) a.f_count[b * gamma + d - 1] = w_d;
      const int64_t o = (b * gamma + d - 1) * W;
      if (have) {
        a.f_parent[o + rank] = p;
        a.f_cand[o + rank] = c;
        a.f_score[o + rank] = f32_key_value(my);
      } else if (lane < W) {
        a.f_parent[o + lane] = -1;
        a.f_cand[o + lane] = -1;
        a.f_score[o + lane] = neg_inf();
      }
    }
    fkey = my;
    fpos = rank;
    np = w_d;
    total += w_d;
    __builtin_amdgcn_wave_barrier();
  }
}

// Algorithm 1 for sequence b, run by one wavefront once the sequence's candidate ids are
// in LDS and, unless kWait, all its score slabs; with kWait the slab of position i is
// awaited before depth i + 1 first reads it.
template <int KT, int R, bool kWait>
__device__ __forceinline__ void fast_search(const TreeArgs& a, const FastSmem& sm, int64_t b, int lane,
                                            uint64_t magic_w) {
  const int gamma = a.gamma, W = a.W;
  const int GW = gamma * W;

  int total = 0;
  expand_depths<KT, R, kWait>(a, sm, b, lane, total);

  // ---- global pruning: Top_budget over the supertree --------------------------------
  const int n_sel = total < a.budget ? total : a.budget;
  if (GW <= 4 * kWave)
    prune_supertree<4>(sm, GW, total, n_sel, lane);
  else if (GW <= 8 * kWave)
    prune_supertree<8>(sm, GW, total, n_sel, lane);
  else
    prune_supertree<16>(sm, GW, total, n_sel, lane);
  // Emission order = rank under (score desc, depth asc, position asc); slot = 1 + rank.
  const int nrows = (n_sel + kWave - 1) / kWave;  // <= 4
  uint2 ent[4];
  int slot[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int i = rb * kWave + lane;
    const uint2 st = sm.stage[i];
    ent[rb] = i < n_sel ? st : make_uint2(0u, 0u);
    slot[rb] = 0;
    if (rb < nrows) {
      slot[rb] = 1 + rank_in_stage(sm.stage, n_sel, order_value(ent[rb].x, ent[rb].y));
      if (i < n_sel) sm.f_slot[~ent[rb].x] = slot[rb];
    }
  }
  __builtin_amdgcn_wave_barrier();

  const int N = a.budget + 1;
  const int words = (N + 31) / 32;
  const int n_nodes = 1 + n_sel;
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
    sm.anc[0] = -1;
  }
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    if (rb < nrows && rb * kWave + lane < n_sel) {
      const int f = static_cast<int>(~ent[rb].x);
      const int d = div_k(f, magic_w) + 1;
      const uint32_t info = sm.s_info[f];
      const int p = static_cast<int>(info & 0xFFFFu);
      const int c = static_cast<int>(info >> 16);
      const int ps = d == 1 ? 0 : sm.f_slot[(d - 2) * W + p];
      const int s = slot[rb];
      tok[s] = sm.cids[(d - 1) * KT + c];
      par[s] = ps;
      dep[s] = d;
      crk[s] = c;
      scr[s] = f32_key_value(ent[rb].y);
      sm.anc[s] = ps;
    }
  }
  for (int n = n_nodes + lane; n < N; n += kWave) {
    tok[n] = -1;
    par[n] = -1;
    dep[n] = -1;
    crk[n] = -1;
    scr[n] = neg_inf();
  }
  __builtin_amdgcn_wave_barrier();

  // ---- ancestor mask by pointer jumping ------------------------------------------------
  // After round k, m covers the node and its 2^k - 1 nearest ancestors and `up` points
  // 2^k steps up; a chain has at most gamma + 1 nodes.
  if (a.mask) {
    const int mrows = (N + kWave - 1) / kWave;  // <= 4
    uint32_t m[4][kMaskWords];
    int up[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int n = rb * kWave + lane;
      const bool live = rb < mrows && n < n_nodes;
      const int an = sm.anc[n < n_nodes ? n : 0];
      up[rb] = live ? an : -1;
#pragma unroll
      for (int w = 0; w < kMaskWords; ++w) m[rb][w] = (live && (n >> 5) == w) ? (1u << (n & 31)) : 0u;
    }
    int rounds = 0;
    while ((1 << rounds) < gamma + 1) ++rounds;
    for (int it = 0; it < rounds; ++it) {
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        const int n = rb * kWave + lane;
        if (rb < mrows && n < n_nodes) {
          uint4* dst = reinterpret_cast<uint4*>(sm.mk + n * kMaskWords);
          dst[0] = make_uint4(m[rb][0], m[rb][1], m[rb][2], m[rb][3]);
          dst[1] = make_uint4(m[rb][4], m[rb][5], m[rb][6], m[rb][7]);
          sm.anc[n] = up[rb];
        }
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        if (rb < mrows && up[rb] >= 0) {
          const uint4* src = reinterpret_cast<const uint4*>(sm.mk + up[rb] * kMaskWords);
          const uint4 lo = src[0], hi = src[1];
          m[rb][0] |= lo.x;
          m[rb][1] |= lo.y;
          m[rb][2] |= lo.z;
          m[rb][3] |= lo.w;
          m[rb][4] |= hi.x;
          m[rb][5] |= hi.y;
          m[rb][6] |= hi.z;
          m[rb][7] |= hi.w;
          up[rb] = sm.anc[up[rb]];
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    uint32_t* mrow = a.mask + b * static_cast<int64_t>(N) * words;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int n = rb * kWave + lane;
      if (rb < mrows && n < N) {
#pragma unroll
        for (int w = 0; w < kMaskWords; ++w)
          if (w < words) mrow[n * words + w] = m[rb][w];
      }
    }
  }
}

template <int KT, int R>
__global__ __launch_bounds__(kWave) void build_tree_fast_kernel(TreeArgs a, uint64_t magic_w) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int lane = threadIdx.x;
  const int64_t b = blockIdx.x;
  const int gamma = a.gamma;
  const FastSmem sm = fast_smem(smem_raw, fast_layout(gamma, KT, a.W));
  // Stage this sequence's score slabs and candidate ids.
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
  const int32_t* gids = a.cand_ids + b * gamma * KT;
  for (int e = lane; e < gamma * KT; e += kWave) sm.cids[e] = gids[e];
  __syncthreads();
  slab_row_max<KT>(sm.slab, sm.rmax, lane, gamma * KT, kWave);
  __syncthreads();
  fast_search<KT, R, false>(a, sm, b, lane, magic_w);
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
    if (a.K == 4)
      UBT_FAST_ROWS(4);
    else if (a.K == 8)
      UBT_FAST_ROWS(8);
    else
      UBT_FAST_ROWS(16);
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
  return feat_dtype == 1 && fast_tree_fits(gamma, K, W);
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

hipError_t launch_tree_mask(const int32_t* parent, const int32_t* n_nodes, int B, int N, uint32_t* mask,
                            hipStream_t stream) {
  hipLaunchKernelGGL(tree_mask_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0, stream, parent, n_nodes, N,
                     mask);
  return hipGetLastError();
}

}  // namespace ubt
