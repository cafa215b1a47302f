// The tree search of the one-launch draft step, split over two waves of a sequence's
// workgroup (Appendix A, Algorithm 1: Eqs. ubtree-frontier and ubtree-pruning; the mask
// of Appendix A / Verification via Tree-attention).
//
// The search wave runs the depth-wise expansion F_d = Top_W(E_d) with the frontier held
// one entry per lane, like the register-resident search, but it lays out E_d by the
// parents' positions in its own compacted stage (stage order) rather than by their rank
// in F_{d-1}.  The ranks only decide exact ties: the order within a depth is score desc,
// then the parent's rank in F_{d-1}, then the candidate rank, i.e. (key desc, true index
// asc) with true index = rank(parent) * K + c.  The selected set does not depend on that
// index unless keys tie exactly at the Top_W boundary, so the search wave needs the ranks
// only then (it waits for them) and never ranks F_d itself.
//
// The pruner wave takes each published stage, ranks its entries under the true order,
// stores F_d in rank order (score key, parent rank and candidate rank, as the beam kernel
// does) and publishes the ranks, so ranking and storing F_d are off the search wave's
// chain.  After the last depth every wave of the workgroup takes part in the global
// pruning, the emission and the mask.
//
// Stages and ranks pass through rings of kPipeRing buffers; the search wave writes the
// stage of depth d only after the pruner has taken the stage of depth d - kPipeRing.
// Every wait is bounded (a timeout sets the workgroup's fail word).
#pragma once

#include "search.h"

namespace ubt {
namespace {

constexpr int kPipeRing = 4;
constexpr int kFinishSurv = 256;  // survivors the finish ranks by counting (else the general path)
constexpr int kPipeStageLive = kFastMaxW + 16;             // up to W live entries + 16 zero entries
constexpr int kPipeStageCap = kPipeStageLive + kWave;      // + one dummy slot per lane

struct PipeSearchLayout {
  uint32_t stage, rank, stage_ready, rank_ready, fbuf, misc, total;
};

__host__ __device__ inline PipeSearchLayout pipe_search_layout(uint32_t base, int gamma) {
  PipeSearchLayout L{};
  uint32_t p = base;
  auto take = [&p](size_t bytes) {
    const uint32_t at = p;
    p += static_cast<uint32_t>((bytes + 15) & ~static_cast<size_t>(15));
    return at;
  };
  L.stage = take(static_cast<size_t>(kPipeRing) * kPipeStageCap * sizeof(uint2));
  L.rank = take(static_cast<size_t>(kPipeRing) * kWave * sizeof(int32_t));
  L.stage_ready = take(static_cast<size_t>(gamma) * sizeof(uint32_t));
  L.rank_ready = take(static_cast<size_t>(gamma) * sizeof(uint32_t));
  L.fbuf = take((kWave + 16) * sizeof(uint2));    // stage entries (+16 zero entries) for ranking
  L.misc = take(4 * sizeof(uint32_t));            // the supertree's node count, the finish's survivor count
  L.total = p;
  return L;
}

struct PipeSearchSmem {
  uint2* stage;           // [kPipeRing][kPipeStageCap]: (~layout index, key), stage order
  int32_t* rank;          // [kPipeRing][64]: rank in F_d of stage position j
  uint32_t* stage_ready;  // [gamma]
  uint32_t* rank_ready;   // [gamma]
  uint2* fbuf;            // [80]: F_d's (~true index, key) in stage order, then 16 zero entries
  uint32_t* misc;         // [4]: the supertree's node count (pruner -> every wave), the finish's survivors
};

__device__ __forceinline__ PipeSearchSmem pipe_search_smem(unsigned char* raw, const PipeSearchLayout& L) {
  PipeSearchSmem ps;
  ps.stage = reinterpret_cast<uint2*>(raw + L.stage);
  ps.rank = reinterpret_cast<int32_t*>(raw + L.rank);
  ps.stage_ready = reinterpret_cast<uint32_t*>(raw + L.stage_ready);
  ps.rank_ready = reinterpret_cast<uint32_t*>(raw + L.rank_ready);
  ps.fbuf = reinterpret_cast<uint2*>(raw + L.fbuf);
  ps.misc = reinterpret_cast<uint32_t*>(raw + L.misc);
  return ps;
}

__device__ __forceinline__ void publish_flag(uint32_t* f) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __hip_atomic_store(f, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// The search wave: depth-wise expansion over the slabs the helper waves publish.
template <int KT, int R>
__device__ __forceinline__ void pipe_search_wave(const TreeArgs& a, const FastSmem& sm, const PipeSearchSmem& ps,
                                                 int lane) {
  constexpr int kLogK = KT == 4 ? 2 : (KT == 8 ? 3 : 4);
  const int gamma = a.gamma, W = a.W;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  uint32_t fkey = f32_key(0.f);
  float nq[KT];
  wait_slab(sm, 0, t0);
  load_row<KT>(sm.slab, nq);  // depth 1 extends the root through row 0
  float rm = sm.rmax[0];
  int np = 1;
  const float zeta = a.zeta;
  const bool with_zeta = zeta != 0.f;
  for (int d = 1; d <= gamma; ++d) {
    // Children of stage entry j (lane j) go to layout index j * K + c.
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
      float4* dst = reinterpret_cast<float4*>(sm.xpose + lane * KT);
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
    // Top_W on the keys; the boundary is exact unless keys tie there.
    uint64_t sel[R];
    uint32_t t = 0u;
    bool exact = true;
    {
      uint32_t kmax, kmin;
      if (np >= W) {
        kmax = wave_umax(best_key);
        kmin = wave_umin(lane < np ? best_key : ~0u);
      } else {
        uint32_t hi = 0, lo = ~0u;
#pragma unroll
        for (int r = 0; r < R; ++r) {
          hi = max(hi, key[r]);
          lo = min(lo, key[r] != 0u ? key[r] : ~0u);
        }
        kmax = wave_umax(hi);
        kmin = wave_umin(lo);
      }
      if (n <= w_d) {
#pragma unroll
        for (int r = 0; r < R; ++r) sel[r] = ballot(key[r] != 0u);
      } else {
        t = kmax;
        exact = false;
        if (kmax != kmin) {
          uint32_t m = 0x80000000u >> __clz(kmax ^ kmin);
          t = kmax & ~(m | (m - 1u));
          int cnt;
          do {
            const uint32_t cand = t | m;
            cnt = 0;
#pragma unroll
            for (int r = 0; r < R; ++r) {
              sel[r] = ballot(key[r] >= cand);
              cnt += popc(sel[r]);
            }
            t = cnt > w_d ? cand : t;
            m = radix_next(m, cnt, w_d, 0u);
          } while (m != 0u);
          exact = cnt == w_d;
        }
      }
    }
    if (!exact) {
      // Keys tie at the boundary t: take every key above t, then the tied entries of
      // smallest true index, which needs the ranks of F_{d-1}.
      if (d > 1) wait_flag(&ps.rank_ready[d - 2], sm.fail, t0);
      const int32_t* prk = ps.rank + ((d - 2) & (kPipeRing - 1)) * kWave;
      int left = w_d;
      uint64_t eq[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        sel[r] = ballot(key[r] > t);
        left -= popc(sel[r]);
        eq[r] = ballot(key[r] == t);
      }
      uint32_t tidx[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int e = r * kWave + lane;
        tidx[r] = d == 1 ? static_cast<uint32_t>(e)
                         : (static_cast<uint32_t>(prk[(e >> kLogK) & (kWave - 1)]) << kLogK) |
                               static_cast<uint32_t>(e & (KT - 1));
      }
      for (; left > 0; --left) {
        uint32_t lo = ~0u;
#pragma unroll
        for (int r = 0; r < R; ++r) lo = min(lo, lane_in(eq[r]) ? tidx[r] : ~0u);
        const uint32_t mn = wave_umin(lo);
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const uint64_t hit = ballot(lane_in(eq[r]) && tidx[r] == mn);
          sel[r] |= hit;
          eq[r] &= ~hit;
        }
      }
    }
    // The stage buffer of depth d is free once the pruner has taken depth d - kPipeRing.
    if (d > kPipeRing) wait_flag(&ps.rank_ready[d - 1 - kPipeRing], sm.fail, t0);
    uint2* stg = ps.stage + ((d - 1) & (kPipeRing - 1)) * kPipeStageCap;
    {
      const int dummy = kPipeStageLive + lane;
      int pos = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int at = lane_in(sel[r]) ? pos + static_cast<int>(lanes_below(sel[r])) : dummy;
        stg[at] = make_uint2(~static_cast<uint32_t>(r * kWave + lane), key[r]);
        pos += popc(sel[r]);
      }
      stg[lane < 16 ? w_d + lane : dummy] = make_uint2(0u, 0u);
    }
    publish_flag(&ps.stage_ready[d - 1]);
    const uint2 st = stg[lane];
    const bool have = lane < w_d;
    const int e = have ? static_cast<int>(~st.x) : 0;
    const int c = e & (KT - 1);
    if (d < gamma) {
      wait_slab(sm, d, t0);
      load_row<KT>(sm.slab + (d * KT + c) * KT, nq);
      rm = sm.rmax[d * KT + c];
    }
    fkey = have ? st.y : 0u;
    np = w_d;
    __builtin_amdgcn_wave_barrier();
  }
}

// The pruner wave: ranks each F_d as it is published and stores it in rank order, then
// leaves the supertree's node count for finish_tree_coop.
template <int KT>
__device__ __forceinline__ void pipe_prune_wave(const TreeArgs& a, const FastSmem& sm, const PipeSearchSmem& ps,
                                                int lane) {
  constexpr int kLogK = KT == 4 ? 2 : (KT == 8 ? 3 : 4);
  const int gamma = a.gamma, W = a.W;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  int prev_rank = 0;  // rank in F_{d-1} of stage position `lane`
  int np = 1;
  int total = 0;
  for (int d = 1; d <= gamma; ++d) {
    const int n = np * KT;
    const int w_d = n < W ? n : W;
    wait_flag(&ps.stage_ready[d - 1], sm.fail, t0);
    const uint2 st = ps.stage[((d - 1) & (kPipeRing - 1)) * kPipeStageCap + lane];
    const bool have = lane < w_d;
    const uint32_t e = have ? ~st.x : 0u;
    const uint32_t key = have ? st.y : 0u;
    // True index: the parent's rank in F_{d-1} (from its stage position), then c.
    const int pr = d == 1 ? 0 : __shfl(prev_rank, static_cast<int>(e >> kLogK));
    const uint32_t tidx = (static_cast<uint32_t>(pr) << kLogK) | (e & (KT - 1));
    const uint2 mine = have ? make_uint2(~tidx, key) : make_uint2(0u, 0u);
    ps.fbuf[lane] = mine;
    if (lane < 16) ps.fbuf[w_d + lane] = make_uint2(0u, 0u);
    __builtin_amdgcn_wave_barrier();
    const int rank = rank_in_stage(ps.fbuf, w_d, order_value(mine.x, mine.y));
    if (have) ps.rank[((d - 1) & (kPipeRing - 1)) * kWave + lane] = rank;
    publish_flag(&ps.rank_ready[d - 1]);
    // F_d in rank order: score key, parent rank and candidate rank.
    const int fb = (d - 1) * W;
    if (have) {
      sm.s_key[fb + rank] = key;
      sm.s_info[fb + rank] = static_cast<uint32_t>(pr) | (static_cast<uint32_t>(e & (KT - 1)) << 16);
    } else if (lane < W) {
      sm.s_key[fb + lane] = 0u;
    }
    prev_rank = rank;
    np = w_d;
    total += w_d;
    __builtin_amdgcn_wave_barrier();
  }
  if (lane == 0) ps.misc[0] = static_cast<uint32_t>(total);
}

// Global pruning (Eq. ubtree-pruning), emission and the mask, by every wave of the
// workgroup once the pruner has stored the whole supertree.  The entries at or above a
// lower bound of the budget-th key (the survivors) are ranked by counting, one thread
// per survivor: rank < budget selects Top_budget and is the emission order at once.
// Node writes and the mask's rows (each a walk up the parent slots) are spread over all
// threads.  Every wave of the workgroup must call it.
template <int KT>
__device__ __forceinline__ void finish_tree_coop(const TreeArgs& a, const FastSmem& sm, const PipeSearchSmem& ps,
                                                 int64_t b, int w, int nw, int lane, uint64_t magic_w) {
  const int gamma = a.gamma, W = a.W, budget = a.budget;
  const int GW = gamma * W;
  const int tid = static_cast<int>(threadIdx.x), nthreads = static_cast<int>(blockDim.x);
  // The rank ring and the children's transpose buffer are free once every wave has
  // arrived (the pruner writes the ring up to its last depth).
  uint32_t* n_surv = ps.misc + 1;                            // the survivor count
  int32_t* srank = reinterpret_cast<int32_t*>(sm.xpose);     // rank of each staged entry
  if (tid == 0) *n_surv = 0u;                                // only the finish uses misc[1]
  __syncthreads();
  const int total = static_cast<int>(ps.misc[0]);
  const int n_sel = total < budget ? total : budget;
  // A lower bound of the n_sel-th largest key: the smallest key of the shallowest depths
  // that hold n_sel entries together (depth d holds w_d = min(w_{d-1} K, W) of them).
  int fcut = 0;
  {
    int np = 1, cum = 0;
    for (int d = 1; d <= gamma && cum < n_sel; ++d) {
      const int n = np * KT;
      np = n < W ? n : W;
      cum += np;
      fcut = d * W;
    }
  }
  // Every wave takes the bound itself (a few dozen keys), so no barrier is needed before
  // the survivors are staged.
  uint32_t lo = ~0u;
  for (int f = lane; f < fcut; f += kWave) {
    const uint32_t k = sm.s_key[f];
    lo = k != 0u ? min(lo, k) : lo;
  }
  const uint32_t bound = wave_umin(lo);
  // The survivors (keys at or above the bound) hold Top_budget; they are staged as
  // (~flat index, key) in any order.
  for (int f0 = 0; f0 < GW; f0 += nthreads) {
    const int f = f0 + tid;
    const uint32_t k = f < GW ? sm.s_key[f] : 0u;
    const bool in = k != 0u && k >= bound;
    const uint64_t m = ballot(in);
    uint32_t at = 0u;
    if (lane == 0 && m != 0ull)
      at = atomicAdd(n_surv, static_cast<uint32_t>(popc(m)));
    const int pos = static_cast<int>(__builtin_amdgcn_readlane(at, 0)) + static_cast<int>(lanes_below(m));
    if (in && pos < kFinishSurv) sm.stage[pos] = make_uint2(~static_cast<uint32_t>(f), k);
  }
  __syncthreads();
  int n_stage = static_cast<int>(*n_surv);
  if (n_stage <= kFinishSurv) {
    // Rank of each survivor under (score desc, depth asc, rank asc): the selection is
    // rank < n_sel, and the rank is its emission order.
    // Four lanes per survivor, lane q of the quad counting the pairs j = 2 q, 2 q + 8, ...
    // (two entries per 16-byte load).
    const uint4* s4 = reinterpret_cast<const uint4*>(sm.stage);
    const int q = tid & 3;
    for (int i0 = tid >> 2; i0 < n_stage; i0 += nthreads >> 2) {  // the same for a quad's lanes
      const uint2 me = sm.stage[i0];
      const uint64_t mv = order_value(me.x, me.y);
      int a0 = 0, a1 = 0;
#pragma unroll 4
      for (int j = 2 * q; j < n_stage; j += 8) {
        const uint4 o = s4[j >> 1];
        a0 += order_value(o.x, o.y) > mv ? 1 : 0;
        a1 += (j + 1 < n_stage && order_value(o.z, o.w) > mv) ? 1 : 0;
      }
      const int ahead = quad_sum(a0 + a1);
      if (q == 0) {
        srank[i0] = ahead;
        if (ahead < n_sel) sm.f_slot[~me.x] = 1 + ahead;
      }
    }
  } else {
    // Many equal keys at the bound: wave 0 selects Top_budget (prune_supertree), then the
    // emission ranks are counted chunk by chunk, each 16-entry chunk of the selection
    // scanned by one wave for every selected entry (LDS adds combine the counts).
    int32_t* erank = ps.rank;
    for (int i = tid; i < kPipeRing * kWave; i += nthreads) erank[i] = 0;
    if (w == 0) {
      if (GW <= 4 * kWave)
        prune_supertree<4>(sm, GW, total, n_sel, lane);
      else if (GW <= 8 * kWave)
        prune_supertree<8>(sm, GW, total, n_sel, lane);
      else
        prune_supertree<16>(sm, GW, total, n_sel, lane);
    }
    __syncthreads();
    const int nrows = (n_sel + kWave - 1) / kWave;  // <= 4
    uint64_t mine[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int i = rb * kWave + lane;
      const uint2 st = sm.stage[i < n_sel ? i : 0];
      mine[rb] = i < n_sel ? order_value(st.x, st.y) : ~0ull;
    }
    const uint4* s4 = reinterpret_cast<const uint4*>(sm.stage);
    for (int ch = w; ch < (n_sel + 15) / 16; ch += nw) {
      uint4 v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = s4[ch * 8 + i];
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        if (rb < nrows) {
          int c0 = 0, c1 = 0;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            c0 += order_value(v[i].x, v[i].y) > mine[rb] ? 1 : 0;
            c1 += order_value(v[i].z, v[i].w) > mine[rb] ? 1 : 0;
          }
          const int cnt = c0 + c1;
          if (rb * kWave + lane < n_sel && cnt) atomicAdd(&erank[rb * kWave + lane], cnt);
        }
      }
    }
    __syncthreads();
    for (int i = tid; i < n_sel; i += nthreads) {
      srank[i] = erank[i];
      sm.f_slot[~sm.stage[i].x] = 1 + erank[i];
    }
    n_stage = n_sel;
  }
  __syncthreads();
  const int N = budget + 1;
  const int words = (N + 31) / 32;
  const int n_nodes = 1 + n_sel;
  int32_t* tok = a.token + b * N;
  int32_t* par = a.parent + b * N;
  int32_t* dep = a.depth + b * N;
  int32_t* crk = a.cand_rank + b * N;
  float* scr = a.score + b * N;
  // A wait of this workgroup that ran out of time leaves scores that were never
  // published behind the tree: the sequence is then marked with n_nodes = 0, and the
  // launch's error word is set.
  const bool failed =
      __builtin_amdgcn_readfirstlane(__hip_atomic_load(sm.fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) != 0u;
  if (tid == 0) {
    a.n_nodes[b] = failed ? 0 : n_nodes;
    if (failed && a.err) __hip_atomic_store(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    tok[0] = a.anchor[b];
    par[0] = -1;
    dep[0] = 0;
    crk[0] = -1;
    scr[0] = 0.f;
    sm.anc[0] = -1;
  }
  for (int i = tid; i < n_stage; i += nthreads) {
    if (srank[i] >= n_sel) continue;
    const uint2 st = sm.stage[i];
    const int f = static_cast<int>(~st.x);
    const int d = div_k(f, magic_w) + 1;
    const uint32_t info = sm.s_info[f];
    const int p = static_cast<int>(info & 0xFFFFu);
    const int c = static_cast<int>(info >> 16);
    const int ps_ = d == 1 ? 0 : sm.f_slot[(d - 2) * W + p];
    const int slot = 1 + srank[i];
    tok[slot] = sm.cids[(d - 1) * KT + c];
    par[slot] = ps_;
    dep[slot] = d;
    crk[slot] = c;
    scr[slot] = f32_key_value(st.y);
    sm.anc[slot] = ps_;
  }
  for (int nn = n_nodes + tid; nn < N; nn += nthreads) {
    tok[nn] = -1;
    par[nn] = -1;
    dep[nn] = -1;
    crk[nn] = -1;
    scr[nn] = neg_inf();
  }
  __syncthreads();
  if (a.mask) {
    // Row n: the node and its ancestors, by walking the parent slots (a chain of at most
    // gamma + 1 nodes; parents precede children, so every step decreases).
    uint32_t* mrow = a.mask + b * static_cast<int64_t>(N) * words;
    for (int nn = tid; nn < N; nn += nthreads) {
      uint32_t wv[kMaskWords] = {0, 0, 0, 0, 0, 0, 0, 0};
      if (nn < n_nodes) {
        int m = nn;
        for (int step = 0; step <= gamma && m >= 0; ++step) {
          const uint32_t bit = 1u << (m & 31);
          const int wi = m >> 5;
#pragma unroll
          for (int k = 0; k < kMaskWords; ++k) wv[k] |= (k == wi) ? bit : 0u;
          m = sm.anc[m];
        }
      }
#pragma unroll
      for (int k = 0; k < kMaskWords; ++k)
        if (k < words) mrow[nn * words + k] = wv[k];
    }
  }
}

}  // namespace
}  // namespace ubt
