// Register-resident tree search (Appendix A, Algorithm 1) for the common shapes, shared
// by the search kernels and the one-launch draft step: depth-wise expansion (Eq.
// ubtree-frontier), global pruning (Eq. ubtree-pruning) and the ancestor mask.
#pragma once

#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

constexpr int kMaxNodes = 256;

// e / K for 0 <= e < 2^16 and 1 <= K <= 64, with magic = ceil(2^32 / K).
__device__ __forceinline__ int div_k(int e, uint64_t magic) {
  return static_cast<int>((static_cast<uint64_t>(static_cast<uint32_t>(e)) * magic) >> 32);
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
constexpr int kFastMaxWK = 1024;
constexpr int kFastMaxGW = 1024;
constexpr int kFastMaxW = 64;
constexpr int kStageLive = 272;                // up to 255 selected entries + 16 zero entries
constexpr int kStageCap = kStageLive + kWave;  // + one dummy slot per lane
constexpr int kMaskWords = 8;                  // ceil(256 / 32)
constexpr int kBoundWords = 32;                // K = 64: per-parent best keys (16), per-wave counts

struct FastLayout {
  uint32_t slab, rmax, cids, xpose, stage, s_key, s_info, f_slot, anc, mk, ready, fail, bound, total;
};

__host__ __device__ inline FastLayout fast_layout(int gamma, int K, int W) {
  FastLayout L{};
  uint32_t p = 0;
  auto take = [&p](size_t bytes) {
    const uint32_t at = p;
    p += static_cast<uint32_t>((bytes + 15) & ~static_cast<size_t>(15));
    return at;
  };
  // K = 64: the slabs (gamma K^2 floats) do not fit; two depths' slabs at a time are staged.
  const bool in_lds = K <= 16;
  L.slab = take((in_lds ? static_cast<size_t>(gamma) : 2) * K * K * sizeof(float));
  L.rmax = take(in_lds ? static_cast<size_t>(gamma) * K * sizeof(float) : 0);
  L.cids = take(static_cast<size_t>(gamma) * K * sizeof(int32_t));
  // K = 64: the survivors' stage (up to W K entries, 16 zero entries, a dummy per lane).
  L.xpose = take(K <= 16 ? kFastMaxWK * sizeof(float) : (kFastMaxWK + 16 + kWave) * sizeof(uint2));
  L.stage = take(kStageCap * sizeof(uint2));
  L.s_key = take(static_cast<size_t>(gamma) * W * sizeof(uint32_t));
  L.s_info = take(static_cast<size_t>(gamma) * W * sizeof(uint32_t));
  L.f_slot = take(static_cast<size_t>(gamma) * W * sizeof(int32_t));
  L.anc = take(kMaxNodes * sizeof(int32_t));
  L.mk = take(kMaxNodes * kMaskWords * sizeof(uint32_t));
  L.ready = take(static_cast<size_t>(gamma) * sizeof(uint32_t));
  L.fail = take(sizeof(uint32_t));
  L.bound = take(kBoundWords * sizeof(uint32_t));
  L.total = p;
  return L;
}

__host__ __device__ inline bool fast_tree_fits(int gamma, int K, int W) {
  const bool shape = ((K == 4 || K == 8 || K == 16) && W * K <= 512) || (K == 64 && W * K <= kFastMaxWK);
  return shape && W <= kFastMaxW && gamma * W <= kFastMaxGW;
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
  // Four independent counts: on a lone wave, one running count would make every
  // compare-and-add wait for the previous one.
  int acc[4] = {0, 0, 0, 0};
  for (int ch = 0; ch < chunks; ++ch) {
    uint4 nxt[8];
    if (ch + 1 < chunks) {
#pragma unroll
      for (int i = 0; i < 8; ++i) nxt[i] = s4[(ch + 1) * 8 + i];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      acc[i & 3] += order_value(cur[i].x, cur[i].y) > mine ? 1 : 0;
      acc[i & 3] += order_value(cur[i].z, cur[i].w) > mine ? 1 : 0;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) cur[i] = nxt[i];
  }
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
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
  uint32_t* ready;  // per position: its slab is in LDS (one-launch kernels only)
  uint32_t* fail;   // nonzero once a wait of this workgroup ran out of time (one-launch kernels only)
  uint32_t* bound;  // K = 64: [0, 16) best child key per parent, [16, 20) survivors per wave
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
  sm.fail = reinterpret_cast<uint32_t*>(raw + L.fail);
  sm.bound = reinterpret_cast<uint32_t*>(raw + L.bound);
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

// Bound of every wait inside a launch: 1 s of the 100 MHz real-time counter.  The
// producers a wait depends on run unconditionally in the same launch, so the bound is
// only reached on a stalled device; the wait then reports failure instead of spinning on.
constexpr uint64_t kWaitTicks = 100000000ull;

// Waits until the workgroup-scope flag *f is set by another wave of the same workgroup.
// Returns false if the wait ran out of time (t0: the waiting wave's start time); the
// workgroup's fail word is then set.
__device__ __forceinline__ bool wait_flag(uint32_t* f, uint32_t* fail, uint64_t t0) {
  for (;;) {
    const uint32_t v = __hip_atomic_load(f, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
    if (__builtin_amdgcn_readfirstlane(v) != 0u) return true;
    if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) {
      __hip_atomic_store(fail, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      return false;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Waits until slab i has been published.
__device__ __forceinline__ bool wait_slab(const FastSmem& sm, int i, uint64_t t0) {
  return wait_flag(&sm.ready[i], sm.fail, t0);
}

// Relaxed agent-scope accesses: they go to and come from the device-coherent level, so a
// workgroup on another XCD (with its own L2) sees them.
__device__ __forceinline__ uint32_t agent_load_u32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void agent_store_u32(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until the agent-scope word *f, set by another workgroup of the same launch, is
// nonzero.  The wave's later loads are issued only after this load has returned (the loop
// exits on its value).  Returns false if the wait ran out of time; the workgroup's fail
// word is then set.
__device__ __forceinline__ bool wait_agent_word(const uint32_t* f, uint32_t* fail, uint64_t t0) {
  for (;;) {
    if (__builtin_amdgcn_readfirstlane(agent_load_u32(f)) != 0u) break;
    if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) {
      __hip_atomic_store(fail, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      return false;
    }
    __builtin_amdgcn_s_sleep(2);
  }
  __atomic_signal_fence(__ATOMIC_SEQ_CST);  // no load is moved above the wait
  return true;
}

// Ancestor mask of a tree whose slots 0..n_nodes-1 are in `anc` (anc[n] = parent slot,
// anc[0] = -1), by pointer jumping: after round k, a node's mask covers it and its
// 2^k - 1 nearest ancestors and `up` points 2^k steps up; a chain of at most
// max_depth + 1 nodes needs ceil(log2(max_depth + 1)) rounds.  Writes rows 0..N-1 of
// mrow ([N, ceil(N/32)] words; rows >= n_nodes zero).  anc and mk (kMaxNodes rows of
// kMaskWords words) are overwritten.  Run by one whole wavefront.
__device__ __forceinline__ void ancestor_mask(int32_t* anc, uint32_t* mk, int n_nodes, int N, int max_depth,
                                              uint32_t* mrow, int lane) {
  const int words = (N + 31) / 32;
  const int mrows = (N + kWave - 1) / kWave;  // <= 4
  uint32_t m[4][kMaskWords];
  int up[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int n = rb * kWave + lane;
    const bool live = rb < mrows && n < n_nodes;
    const int an = anc[n < n_nodes ? n : 0];
    up[rb] = live ? an : -1;
#pragma unroll
    for (int w = 0; w < kMaskWords; ++w) m[rb][w] = (live && (n >> 5) == w) ? (1u << (n & 31)) : 0u;
  }
  int rounds = 0;
  while ((1 << rounds) < max_depth + 1) ++rounds;
  for (int it = 0; it < rounds; ++it) {
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int n = rb * kWave + lane;
      if (rb < mrows && n < n_nodes) {
        uint4* dst = reinterpret_cast<uint4*>(mk + n * kMaskWords);
        dst[0] = make_uint4(m[rb][0], m[rb][1], m[rb][2], m[rb][3]);
        dst[1] = make_uint4(m[rb][4], m[rb][5], m[rb][6], m[rb][7]);
        anc[n] = up[rb];
      }
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      if (rb < mrows && up[rb] >= 0) {
        const uint4* src = reinterpret_cast<const uint4*>(mk + up[rb] * kMaskWords);
        const uint4 lo = src[0], hi = src[1];
        m[rb][0] |= lo.x;
        m[rb][1] |= lo.y;
        m[rb][2] |= lo.z;
        m[rb][3] |= lo.w;
        m[rb][4] |= hi.x;
        m[rb][5] |= hi.y;
        m[rb][6] |= hi.z;
        m[rb][7] |= hi.w;
        up[rb] = anc[up[rb]];
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
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

// F_d, once selected: the w_d entries of `key` marked in `sel` (entry index e = parent
// position in F_{d-1} * K + candidate rank), compacted to the stage in index order.
// Returns this lane's entry (lane < w_d): its key, parent position p and candidate c.
template <int R, int kLogK>
__device__ __forceinline__ bool frontier_entry(const FastSmem& sm, const uint32_t (&key)[R], const uint64_t (&sel)[R],
                                               int w_d, int lane, uint32_t& mx, uint32_t& my, int& p, int& c) {
  compact_selected<R>(sm.stage, key, sel, w_d, lane);
  const uint2 st = sm.stage[lane];
  const bool have = lane < w_d;
  mx = have ? st.x : 0u;
  my = have ? st.y : 0u;
  const int e = have ? static_cast<int>(~mx) : 0;
  p = e >> kLogK;
  c = e & ((1 << kLogK) - 1);
  return have;
}

// Stores F_d in rank order (score desc, then index) to s_key / s_info (parent = its
// position in F_{d-1}, candidate rank), with the supertree outputs if asked: the lanes
// with `have` hold the w_d entries, each with its rank, and slots w_d..W-1 are cleared.
__device__ __forceinline__ void frontier_store(const TreeArgs& a, const FastSmem& sm, int64_t b, int lane, int d,
                                               int w_d, bool have, int rank, uint32_t my, int p, int c) {
  const int gamma = a.gamma, W = a.W;
  const int fb = (d - 1) * W;
  const bool clear = lane >= w_d && lane < W;
  // A lane may both hold an entry and clear a slot (each lane's slot differs from every
  // rank < w_d it may store to).
  if (have) {
    sm.s_key[fb + rank] = my;
    sm.s_info[fb + rank] = static_cast<uint32_t>(p) | (static_cast<uint32_t>(c) << 16);
  }
  if (clear) sm.s_key[fb + lane] = 0u;
  if (a.f_count) {
    if (lane == 0) a.f_count[b * gamma + d - 1] = w_d;
    const int64_t o = (b * gamma + d - 1) * W;
    if (have) {
      a.f_parent[o + rank] = p;
      a.f_cand[o + rank] = c;
      a.f_score[o + rank] = f32_key_value(my);
    }
    if (clear) {
      a.f_parent[o + lane] = -1;
      a.f_cand[o + lane] = -1;
      a.f_score[o + lane] = neg_inf();
    }
  }
}

// Depth-wise expansion (Eq. ubtree-frontier): F_d = Top_W(E_d) for d = 1..gamma, with the
// slabs in LDS (K <= 16).  F_d is ranked (score desc, parent position, candidate rank) as
// it is formed and stored in that order to s_key / s_info (parent = its position in
// F_{d-1}), with the supertree outputs if asked.  total = the number of supertree nodes.
template <int KT, int R, bool kWait>
__device__ __forceinline__ void expand_depths(const TreeArgs& a, const FastSmem& sm, int64_t b, int lane,
                                              int& total) {
  static_assert(KT <= 16, "K = 64 stages its slabs (expand_depths64)");
  constexpr int kLogK = KT == 4 ? 2 : (KT == 8 ? 3 : 4);
  const int gamma = a.gamma, W = a.W;
  // Frontier entry on lane j < np: score key, position in F, and its slab row for the
  // next depth (loaded as soon as the entry's candidate rank is known).
  uint32_t fkey = f32_key(0.f);
  int fpos = 0;
  float nq[KT];
  float rm;
  const uint64_t t0 = kWait ? __builtin_amdgcn_s_memrealtime() : 0ull;
  if (kWait) wait_slab(sm, 0, t0);
  load_row<KT>(sm.slab, nq);  // depth 1 extends the root through row 0
  rm = sm.rmax[0];
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
    uint32_t mx, my;
    int p, c;
    const bool have = frontier_entry<R, kLogK>(sm, key, sel, w_d, lane, mx, my, p, c);
    if (d < gamma) {
      if (kWait) wait_slab(sm, d, t0);
      load_row<KT>(sm.slab + (d * KT + c) * KT, nq);
      rm = sm.rmax[d * KT + c];
    }
    const int rank = rank_in_stage(sm.stage, w_d, order_value(mx, my));
    frontier_store(a, sm, b, lane, d, w_d, have, rank, my, p, c);
    fkey = my;
    fpos = rank;
    np = w_d;
    total += w_d;
    __builtin_amdgcn_wave_barrier();
  }
}

// The same expansion for K = 64 on kK64Waves waves of one workgroup (a lone wave issues
// too slowly for the 64 W entries of a depth).  The slabs (gamma K^2 floats) do not fit
// in LDS: two are staged at a time, each wave loading a quarter of the slab two depths
// ahead into registers while the current one is searched.  Entry (r, lane) of depth d is
// child `lane` of the frontier entry of rank r in F_{d-1} (index r * 64 + lane: index
// order is (parent rank, candidate rank)); wave w holds the parents r = w, w + 4, ...
//
// Selection: each parent's best child is a wave maximum over its register, and the
// smallest of these W maxima is a lower bound of the W-th best entry (they are W distinct
// entries).  The entries at or above that bound (the survivors, typically a few dozen)
// hold F_d; they are compacted to the survivors' stage and each survivor's rank among
// them (score desc, then index) is counted, so the survivors of rank < W are F_d, already
// ranked.  All waves return with the same `total`.
constexpr int kK64Waves = 4;

//
// kWait: the slabs are written by other workgroups of the same launch.  Before loading the
// slab of depth d a wave waits for ready[d - 1] (an agent-scope word its producer sets
// once the slab's agent-scope stores have completed), then loads it with agent-scope
// loads; a wait that runs out of time sets the workgroup's fail word.  t0: the wave's
// start time.
template <int RW, bool vec, bool kWait = false>
__device__ __forceinline__ void expand_depths64(const TreeArgs& a, const FastSmem& sm, int64_t b, int w, int lane,
                                                int& total, const uint32_t* ready = nullptr, uint64_t t0 = 0) {
  static_assert(!(kWait && vec), "waited slabs are loaded word by word");
  constexpr int KT = 64;
  constexpr int kQuarter = KT * KT / kK64Waves;  // floats of a slab staged by one wave
  const int gamma = a.gamma, W = a.W;
  const float* gq = a.logq + b * gamma * KT * KT + w * kQuarter;
  float P[kQuarter / kWave];  // this wave's quarter of a slab, in flight
  auto load_slab = [&](int d) {  // slab of depth d (1-based)
    const float* src = gq + static_cast<int64_t>(d - 1) * KT * KT;
    if constexpr (kWait) {
      wait_agent_word(ready + (d - 1), sm.fail, t0);
      const uint32_t* u = reinterpret_cast<const uint32_t*>(src);
#pragma unroll
      for (int i = 0; i < kQuarter / kWave; ++i) P[i] = __uint_as_float(agent_load_u32(u + i * kWave + lane));
    } else if constexpr (vec) {
#pragma unroll
      for (int i = 0; i < kQuarter / (4 * kWave); ++i) {
        const float4 t = reinterpret_cast<const float4*>(src)[i * kWave + lane];
        P[4 * i] = t.x;
        P[4 * i + 1] = t.y;
        P[4 * i + 2] = t.z;
        P[4 * i + 3] = t.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < kQuarter / kWave; ++i) P[i] = src[i * kWave + lane];
    }
  };
  auto store_slab = [&](int d) {
    float* dst = sm.slab + ((d - 1) & 1) * KT * KT + w * kQuarter;
    if constexpr (vec) {
#pragma unroll
      for (int i = 0; i < kQuarter / (4 * kWave); ++i)
        reinterpret_cast<float4*>(dst)[i * kWave + lane] = make_float4(P[4 * i], P[4 * i + 1], P[4 * i + 2], P[4 * i + 3]);
    } else {
#pragma unroll
      for (int i = 0; i < kQuarter / kWave; ++i) dst[i * kWave + lane] = P[i];
    }
  };
  uint32_t* s_best = sm.bound;
  uint32_t* s_cnt = sm.bound + 16;
  uint2* surv = reinterpret_cast<uint2*>(sm.xpose);  // [0, ns) survivors, then 16 zeros
  const int dummy = kFastMaxWK + 16 + lane;
  load_slab(1);
  store_slab(1);
  if (gamma > 1) load_slab(2);
  lds_barrier();
  int np = 1;
  total = 0;
  const float zeta = a.zeta;
  const bool with_zeta = zeta != 0.f;
  for (int d = 1; d <= gamma; ++d) {
    // Slab d + 1 to LDS (its buffer held slab d - 1, whose reads ended before the last
    // barrier of depth d - 1), then slab d + 2 on its way; the barriers of this depth
    // publish slab d + 1 before depth d + 1 reads it.
    if (d + 1 <= gamma) {
      store_slab(d + 1);
      if (d + 2 <= gamma) load_slab(d + 2);
    }
    const float* slab = sm.slab + ((d - 1) & 1) * KT * KT;
    // F_{d-1}: entry r on lane r (depth 1: the root, score 0, extends through row 0).
    uint32_t pkey = f32_key(0.f), pinfo = 0u;
    if (d > 1 && lane < W) {
      pkey = sm.s_key[(d - 2) * W + lane];
      pinfo = sm.s_info[(d - 2) * W + lane];
    }
    uint32_t key[RW];
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      const int r = i * kK64Waves + w;
      const float base = f32_key_value(__builtin_amdgcn_readlane(pkey, r));
      const int row = static_cast<int>(__builtin_amdgcn_readlane(pinfo, r) >> 16);
      float v = base + slab[row * KT + lane];
      if (with_zeta) v += zeta;
      key[i] = r < np ? f32_key(v) : 0u;
    }
    const int n = np * KT;
    const int w_d = n < W ? n : W;
    // The bound: the smallest best child over the W parents (np = W from depth 2 on).
    uint32_t kbound = 1u;  // keys of live entries are nonzero
    if (np >= W) {
#pragma unroll
      for (int i = 0; i < RW; ++i) {
        const int r = i * kK64Waves + w;
        const uint32_t m = wave_umax(key[i]);
        if (r < np && lane == 0) s_best[r] = m;
      }
      lds_barrier();
      kbound = wave_umin(lane < W ? s_best[lane < W ? lane : 0] : ~0u);
    }
    uint64_t sel[RW];
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      sel[i] = ballot(key[i] >= kbound);
      cnt += popc(sel[i]);
    }
    if (lane == 0) s_cnt[w] = static_cast<uint32_t>(cnt);
    lds_barrier();
    const uint32_t c4 = lane < kK64Waves ? s_cnt[lane < kK64Waves ? lane : 0] : 0u;
    int ns = 0, off = 0;
#pragma unroll
    for (int v = 0; v < kK64Waves; ++v) {
      const int cv = static_cast<int>(__builtin_amdgcn_readlane(c4, v));
      off += v < w ? cv : 0;
      ns += cv;
    }
    // Survivors to surv[0, ns) (each wave at its offset, in any order), then 16 zeros.
    int pos = off;
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      const int r = i * kK64Waves + w;
      const int at = lane_in(sel[i]) ? pos + static_cast<int>(lanes_below(sel[i])) : dummy;
      surv[at] = make_uint2(~static_cast<uint32_t>(r * KT + lane), key[i]);
      pos += popc(sel[i]);
    }
    if (w == 0) surv[lane < 16 ? ns + lane : dummy] = make_uint2(0u, 0u);
    lds_barrier();
    // Survivor j is ranked by lane j % 64 of wave (j / 64) % kK64Waves.
    for (int j0 = w * kWave; j0 < ns; j0 += kK64Waves * kWave) {
      const int j = j0 + lane;
      const bool live = j < ns;
      const uint2 st = surv[live ? j : 0];
      const uint32_t mx = live ? st.x : 0u, my = live ? st.y : 0u;
      const int rank = rank_in_stage(surv, ns, order_value(mx, my));
      const bool have = live && rank < w_d;
      const int e = have ? static_cast<int>(~mx) : 0;
      frontier_store(a, sm, b, w == 0 && j0 == 0 ? lane : kWave, d, w_d, have, rank, my, e >> 6, e & (KT - 1));
    }
    np = w_d;
    total += w_d;
    lds_barrier();  // F_d and slab d + 1 published; the survivors and bound words free
  }
}

// Global pruning (Eq. ubtree-pruning), emission and the mask, once the supertree's keys
// and infos are in s_key / s_info (F_d in rank order at (d - 1) * W + rank) and `total`
// counts its nodes.  With kCheckFail, a wait of the workgroup that ran out of time marks
// the sequence with n_nodes = 0 and sets the launch's error word.
template <int KT, bool kCheckFail>
__device__ __forceinline__ void finish_tree(const TreeArgs& a, const FastSmem& sm, int64_t b, int lane,
                                            uint64_t magic_w, int total) {
  const int gamma = a.gamma, W = a.W;
  const int GW = gamma * W;

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
  // A wait of this workgroup that ran out of time (one-launch kernels) leaves scores
  // that were never published behind the tree: the sequence is then marked with
  // n_nodes = 0, and the launch's error word is set if it has one.
  const bool failed =
      kCheckFail && __builtin_amdgcn_readfirstlane(__hip_atomic_load(sm.fail, __ATOMIC_RELAXED,
                                                                     __HIP_MEMORY_SCOPE_WORKGROUP)) != 0u;
  if (lane == 0) {
    a.n_nodes[b] = failed ? 0 : n_nodes;
    if (failed && a.err) __hip_atomic_store(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

  if (a.mask) {
    uint32_t* mrow = a.mask + b * static_cast<int64_t>(N) * words;
    ancestor_mask(sm.anc, sm.mk, n_nodes, N, gamma, mrow, lane);
  }
}

// Algorithm 1 for sequence b, run by one wavefront once the sequence's candidate ids are
// in LDS and, unless kWait, all its score slabs; with kWait the slab of position i is
// awaited before depth i + 1 first reads it.
template <int KT, int R, bool kWait>
__device__ __forceinline__ void fast_search(const TreeArgs& a, const FastSmem& sm, int64_t b, int lane,
                                            uint64_t magic_w) {
  int total = 0;
  expand_depths<KT, R, kWait>(a, sm, b, lane, total);
  finish_tree<KT, kWait>(a, sm, b, lane, magic_w, total);
}

}  // namespace
}  // namespace ubt
