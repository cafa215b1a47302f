// The whole draft step in one launch: softmax statistics and top-K candidates over the
// vocabulary, the selector scores, and the tree search with its ancestor mask.
//
// Method / Unigram Proposer, Eq. (ubtree-unigram) and "Candidate Sets" (per-position LSE
// and C_i); Method / Parallel Computation, Eq. (ubtree-edge-matrix), Depth Calibration,
// Eq. (ubtree-depth), and Appendix A / Path Scores, Eq. (ubtree-path) (log q^bi);
// Appendix A, Algorithm 1 with Eqs. (ubtree-frontier) and (ubtree-pruning) (the tree);
// Appendix A / Verification via Tree-attention (the mask).
//
// The sweep is bound by HBM bandwidth and the search of one sequence is a long chain of
// dependent steps on one wave.  Run one after the other they add up; here they overlap.
// Workgroups 0..B-1 are searchers, one per sequence.  The others stream the logits:
// each of their waves is an independent worker that walks a fixed list of tile tasks
// (one tile = 64 lanes x 4 groups x 16 B), interleaved with every other worker's, so the
// whole chip sweeps the rows in depth-major order and the rows of draft position 1 are
// complete long before those of the last position.  A searcher merges each row of its
// sequence as soon as all of the row's tiles are in, computes that position's score
// slab, and its search wave consumes the slabs in order while later positions stream.
//
// Candidates without a per-row pass: the first S tiles of every row are swept first
// (sample tasks), each keeping its exact top K, and the K-th largest of all their
// candidates becomes the row's threshold (a lower bound of the row's K-th largest
// logit).  Every later tile of the row keeps only its 16-byte groups whose maximum reaches
// the threshold it reads (a few, in fixed slots of its record); a tile that finds no
// threshold yet keeps its exact top K, and one with more such groups than its record
// holds is flagged to be read again.  The merging wave loads every record in a few
// memory round trips, keeps what reaches the final threshold, and selects the row's top
// K, ordered (logit desc, id asc).
//
// Cross-workgroup traffic uses agent-scope (device-coherent) stores and loads, and
// counters are bumped only after the data they cover has completed (s_waitcnt), so no
// cache-wide writeback or invalidation is needed.  Workers never wait on anything; only
// searcher waves wait, each wait bounded in time.  Searchers have the lowest workgroup
// indices, so they are dispatched first and never keep a worker from running.  The
// workspace counters are reset by their last reader, leaving them ready for the next
// launch.
#include "bigram_tile.h"
#include "search.h"
#include "sweep.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

constexpr int kStepWaves = 8;        // waves per workgroup (both roles)
constexpr int kMergeWaves = 4;       // searcher waves 1..4 merge rows and compute slabs
constexpr int kListCap = 576;        // candidates a merging wave collects (one pass adds <= 512)
constexpr uint64_t kWaitTicks = 100000000ull;  // 1 s of the 100 MHz real-time counter

__device__ __forceinline__ void store_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_agent32(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_agent(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t load_agent32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t pack2(uint32_t lo, uint32_t hi) {
  return static_cast<uint64_t>(lo) | (static_cast<uint64_t>(hi) << 32);
}
// Waits until every memory operation issued so far by this wave has completed.
__device__ __forceinline__ void wait_all_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// ---- the task list --------------------------------------------------------------------
// Rows are numbered depth-major: rd = i * B + b for position i of sequence b.  Sample
// tasks (rd, j) for j < S come first, then stream tasks (rd, S + j) for j < nt - S, each
// phase in rd-major order.  Worker g takes tasks g, g + NW, g + 2 NW, ...
struct Task {
  int phase;  // 0 sample, 1 stream, 2 none left
  int rd;
  int j;
};

__device__ __forceinline__ Task task_at(int64_t t, int rows, int S, int NS) {
  const int64_t n_sample = static_cast<int64_t>(rows) * S;
  if (t < n_sample) return Task{0, static_cast<int>(t / S), static_cast<int>(t % S)};
  const int64_t u = t - n_sample;
  if (NS == 0 || u >= static_cast<int64_t>(rows) * NS) return Task{2, 0, 0};
  return Task{1, static_cast<int>(u / NS), static_cast<int>(u % NS)};
}

// ---- workspace and arguments ------------------------------------------------------------
constexpr int kTileGroups = 16;  // groups a tile may hand over; a tile with more is re-read

struct StepArgs {
  const void* logits;
  int64_t V, stride_b, stride_i;
  int B, gamma, K;
  int nt;            // tiles per row
  int S;             // sample tiles per row
  int nw;            // worker waves
  int step0_rd, step0_j;  // NW = step0_rd * S + step0_j
  int step1_rd, step1_j;  // NW = step1_rd * (nt - S) + step1_j
  uint64_t magic_b;  // ceil(2^32 / B)
  int32_t* cand_ids;
  float* cand_logit;
  float* cand_logprob;
  float* lse;
  // Workspace: an error word, then one block per output row holding
  //   done, thr (uint32) at 0: tiles finished, threshold key (0 = none yet);
  //   hdr  [nt][2] uint64 at 16: per tile (max, sum) bits, and (exact entries | groups
  //                    << 8 | re-read flag << 16, K-th key << 32);
  //   ent  [nt][K] uint64 at off_ent: per tile its exact candidates as order values;
  //   grp  [nt][kTileGroups][2] uint64 at off_grp: per tile the 16-byte groups that
  //                    reached the threshold;
  //   gpos [nt][kTileGroups] uint32 at off_gpos: element index of each group's first
  //                    element.
  char* ws;
  uint32_t row_bytes, off_ent, off_grp, off_gpos;
};

constexpr uint32_t kRowBlocks = 256;  // offset of the first row block

__device__ __forceinline__ uint32_t* ws_err(const StepArgs& p) { return reinterpret_cast<uint32_t*>(p.ws); }
__device__ __forceinline__ char* row_block(const StepArgs& p, int orow) {
  return p.ws + kRowBlocks + static_cast<int64_t>(orow) * p.row_bytes;
}
__device__ __forceinline__ uint32_t* row_done(char* blk) { return reinterpret_cast<uint32_t*>(blk); }
__device__ __forceinline__ uint32_t* row_thr(char* blk) { return reinterpret_cast<uint32_t*>(blk + 4); }
__device__ __forceinline__ uint64_t* row_hdr(char* blk) { return reinterpret_cast<uint64_t*>(blk + 16); }
__device__ __forceinline__ uint64_t* row_ent(const StepArgs& p, char* blk) {
  return reinterpret_cast<uint64_t*>(blk + p.off_ent);
}
__device__ __forceinline__ uint64_t* row_grp(const StepArgs& p, char* blk) {
  return reinterpret_cast<uint64_t*>(blk + p.off_grp);
}
__device__ __forceinline__ uint32_t* row_gpos(const StepArgs& p, char* blk) {
  return reinterpret_cast<uint32_t*>(blk + p.off_gpos);
}

// Task fields are wave-uniform; saying so keeps them in scalar registers, so the buffer
// resource of a row is uniform without a waterfall loop around each load.
__device__ __forceinline__ void uniform(Task& c) {
  c.phase = __builtin_amdgcn_readfirstlane(c.phase);
  c.rd = __builtin_amdgcn_readfirstlane(c.rd);
  c.j = __builtin_amdgcn_readfirstlane(c.j);
}

__device__ __forceinline__ void advance(Task& c, const StepArgs& p, int rows) {
  const int S = p.S, NS = p.nt - p.S;
  if (c.phase == 0) {
    c.j += p.step0_j;
    c.rd += p.step0_rd;
    if (c.j >= S) {
      c.j -= S;
      c.rd += 1;
    }
    if (c.rd >= rows) c = task_at(static_cast<int64_t>(c.rd) * S + c.j, rows, S, NS);
  } else if (c.phase == 1) {
    c.j += p.step1_j;
    c.rd += p.step1_rd;
    if (c.j >= NS) {
      c.j -= NS;
      c.rd += 1;
    }
    if (c.rd >= rows) c.phase = 2;
  }
  uniform(c);
}

// Output row (b * gamma + i) of depth-major row rd.
__device__ __forceinline__ int out_row(const StepArgs& p, int rd) {
  const int i = div_k(rd, p.magic_b);
  const int b = rd - i * p.B;
  return b * p.gamma + i;
}

// ---- exact top K of one tile -------------------------------------------------------------
// The tile's n = min(K, elements in the row) largest elements as order values (key desc,
// id asc), lane r holding the r-th; lanes >= n hold 0.
template <typename T>
__device__ __forceinline__ uint64_t tile_topk(const u32x4 (&buf)[kSubGroups], const float (&gmax)[kSubGroups], float lmax,
                              int64_t c0, int64_t V, int K, int lane, WaveLds& s, int& n_out) {
  constexpr int EPG = Traits<T>::kPer;
  // T = the K-th largest lane maximum (0 if fewer than K lanes hold elements): K distinct
  // groups reach it, so it bounds the tile's K-th largest element from below.
  const bool holds = c0 + static_cast<int64_t>(lane) * EPG < V;
  const uint32_t lkey = holds ? Traits<T>::key_value(lmax) : 0u;
  uint32_t* sv = reinterpret_cast<uint32_t*>(s.stage);
  sv[lane] = lkey;
  __builtin_amdgcn_wave_barrier();
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < kWave; j += 4) {
    const uint4 v = *reinterpret_cast<const uint4*>(&sv[j]);
    cnt += (v.x > lkey) + (v.y > lkey) + (v.z > lkey) + (v.w > lkey);
  }
  __builtin_amdgcn_wave_barrier();
  const int n_live = popc(ballot(lkey != 0));
  const uint32_t thr = n_live < K ? 0u : wave_umin(lkey != 0 && cnt < K ? lkey : ~0u);

  // Only groups whose maximum reaches T can hold a top-K element.  They are buffered in
  // LDS (64 at a time), and their elements at or above T go through a window: the best K
  // so far at s.cand[0..held), new ones behind them; when the next chunk might not fit,
  // every entry of the window counts the entries above it and the K best move to their
  // ranks.  Chunks of 64 - K elements keep the window within 64 entries.
  uint32_t pend = passing_groups<T>(gmax, c0, V, thr, false, lane);
  const int chunk = kWave - K;
  int held = 0, fill = 0;
  auto rank_window = [&]() {
    const int cnt = held + fill;
    __builtin_amdgcn_wave_barrier();
    const uint64_t mine = lane < cnt ? s.cand[lane] : 0ull;
    const int r = lane < cnt ? count_above(s.cand, cnt, mine) : kWave;
    __builtin_amdgcn_wave_barrier();
    if (r < K) s.cand[r] = mine;
    __builtin_amdgcn_wave_barrier();
    held = cnt < K ? cnt : K;
    fill = 0;
  };
  while (ballot(pend != 0)) {
    int nbuf = 0;
    pend = buffer_groups<T>(buf, pend, c0, lane, s, nbuf);
    __builtin_amdgcn_wave_barrier();
    const int total = nbuf * EPG;
    for (int e0 = 0; e0 < total; e0 += chunk) {
      const int e = e0 + lane;
      uint64_t v = 0ull;
      bool keep = false;
      if (lane < chunk && e < total) {
        const int g = e / EPG, j = e % EPG;
        const uint32_t word = reinterpret_cast<const uint32_t*>(&s.data[g])[j * 4 / EPG];
        const uint32_t bits = EPG == 8 ? (word >> (16 * (j & 1))) & 0xFFFFu : word;
        const int64_t gid = static_cast<int64_t>(s.base[g]) + j;
        const uint32_t k = Traits<T>::key_bits(bits);
        keep = gid < V && k >= thr;
        v = cand_order(k, static_cast<uint32_t>(gid));
      }
      const uint64_t mk = ballot(keep);
      const int c = popc(mk);
      if (held + fill + c > kWave) rank_window();
      if (keep) s.cand[held + fill + static_cast<int>(lanes_below(mk))] = v;
      fill += c;
    }
    __builtin_amdgcn_wave_barrier();
  }
  rank_window();
  n_out = held;
  const uint64_t out = lane < held ? s.cand[lane] : 0ull;
  __builtin_amdgcn_wave_barrier();
  return out;
}

// ---- workers ------------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void issue_tile(const StepArgs& p, const Task& t, u32x4 (&buf)[kSubGroups], uint32_t& thr,
                                           uint32_t lane_off) {
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * Traits<T>::kPer;
  const int i = div_k(t.rd, p.magic_b);
  const int b = t.rd - i * p.B;
  const T* rp = static_cast<const T*>(p.logits) + b * p.stride_b + i * p.stride_i;
  const __amdgpu_buffer_rsrc_t rsrc = row_resource(rp, static_cast<uint32_t>(p.V * static_cast<int64_t>(sizeof(T))));
  const int tile = t.phase == 0 ? t.j : p.S + t.j;
  load_full<T>(buf, rsrc, tile * SUB, lane_off);
  if (t.phase == 1) thr = load_agent32(row_thr(row_block(p, out_row(p, t.rd))));
}


// Reduces a tile and stores its record: (max, sum), and either the exact top K of the
// tile (sample tiles, and tiles that found no threshold yet) or the groups whose maximum
// reaches thr (up to kTileGroups; a tile with more is flagged to be re-read).
template <typename T, bool kExact>
__device__ __forceinline__ uint64_t process_tile(const StepArgs& p, const Task& t, u32x4 (&buf)[kSubGroups],
                                                 uint32_t thr, int lane, WaveLds& s) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * EPG;
  const int64_t V = p.V;
  const int tile = t.phase == 0 ? t.j : p.S + t.j;
  const int64_t c0 = tile * SUB;
  char* blk = row_block(p, out_row(p, t.rd));
  if (c0 + SUB > V) mask_tail<T>(buf, c0, V, lane);
  float gmax[kSubGroups];
  float lm = neg_inf(), ls = 0.f;
  const float lmax = reduce_sub<T>(buf, gmax, lm, ls);
  const float wm = wave_max(lm);
  const float wsum = wave_sum(lm == neg_inf() ? 0.f : ls * fast_exp2((lm - wm) * kLog2e));
  uint32_t meta = 0u, kth = 0u;
  uint64_t ent = 0ull;
  if (kExact) {
    int n = 0;
    ent = tile_topk<T>(buf, gmax, lmax, c0, V, p.K, lane, s, n);
    const uint32_t last = static_cast<uint32_t>(__shfl(static_cast<int>(ent >> 32), p.K - 1, kWave));
    kth = n == p.K ? __builtin_amdgcn_readfirstlane(last) : 0u;
    meta = static_cast<uint32_t>(n);
    if (lane < n) store_agent(row_ent(p, blk) + tile * p.K + lane, ent);
    if (lane == 0 && kth != 0u) __hip_atomic_fetch_max(row_thr(blk), kth, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    const uint32_t pg = passing_groups<T>(gmax, c0, V, thr, false, lane);
    int ng = 0;
#pragma unroll
    for (int g = 0; g < kSubGroups; ++g) ng += popc(ballot((pg >> g) & 1u));
    if (ng > kTileGroups) {
      meta = 1u << 16;
    } else if (ng > 0) {
      meta = static_cast<uint32_t>(ng) << 8;
      uint64_t* gd = row_grp(p, blk) + tile * kTileGroups * 2;
      uint32_t* gp = row_gpos(p, blk) + tile * kTileGroups;
      int pos = 0;
#pragma unroll
      for (int g = 0; g < kSubGroups; ++g) {
        const bool hit = (pg >> g) & 1u;
        const uint64_t m = ballot(hit);
        if (hit) {
          const int at = pos + static_cast<int>(lanes_below(m));
          store_agent(&gd[2 * at], pack2(buf[g][0], buf[g][1]));
          store_agent(&gd[2 * at + 1], pack2(buf[g][2], buf[g][3]));
          store_agent32(&gp[at], static_cast<uint32_t>(c0) + static_cast<uint32_t>((g * kWave + lane) * EPG));
        }
        pos += popc(m);
      }
    }
  }
  if (lane == 0) {
    uint64_t* hdr = row_hdr(blk) + 2 * tile;
    store_agent(hdr, pack2(__float_as_uint(wm), __float_as_uint(wsum)));
    store_agent(hdr + 1, pack2(meta, kth));
  }
  return ent;
}

// Counts a finished tile of output row `tag`; its record's stores have completed.
__device__ __forceinline__ void count_done(const StepArgs& p, int tag, int lane) {
  if (lane == 0) __hip_atomic_fetch_add(row_done(row_block(p, tag)), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Processes the tile of `cur` (in buf) and puts the next task's tile in flight (into
// nbuf).  A tile that needs its exact top K is processed before the next load is
// issued, so the selection has the registers of both buffers; the other tiles are
// processed while the next one streams in.
//
// When every row has kStepWaves sample tiles, the waves of a workgroup hold the sample
// tiles of one row in the same step (worker g takes task g + k NW, and NW is a multiple
// of kStepWaves), so they pool their top K lists in LDS and wave 0 raises the row's
// threshold to the K-th largest of the pool: a bound from all the sample elements, in
// place before the row's other tiles are read.
template <typename T>
__device__ __forceinline__ void step_tile(const StepArgs& p, const Task& cur, const Task& nxt, u32x4 (&buf)[kSubGroups],
                                          uint32_t thr_in, u32x4 (&nbuf)[kSubGroups], uint32_t& nthr,
                                          uint32_t lane_off, int lane, WaveLds& s, uint64_t* pool, int w) {
  const uint32_t thr = __builtin_amdgcn_readfirstlane(thr_in);
  if (cur.phase == 0 || thr == 0u) {
    const uint64_t ent = process_tile<T, true>(p, cur, buf, 0u, lane, s);
    if (cur.phase == 0 && p.S == kStepWaves) {
      const int K = p.K;
      if (lane < K) pool[w * K + lane] = ent;
      __syncthreads();
      if (w == 0) {
        uint32_t key[2], sub[2];
        uint64_t live[2], sel[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int q = r * kWave + lane;
          const uint64_t v = q < kStepWaves * K ? pool[q] : 0ull;
          key[r] = static_cast<uint32_t>(v >> 32);
          sub[r] = ~static_cast<uint32_t>(v);
          live[r] = ballot(v != 0ull);
        }
        wave_select<2>(key, sub, live, K, 32, sel);
        uint32_t kmin = ~0u;
#pragma unroll
        for (int r = 0; r < 2; ++r) kmin = lane_in(sel[r]) ? min(kmin, key[r]) : kmin;
        const uint32_t tstar = popc(sel[0]) + popc(sel[1]) < K ? 0u : wave_umin(kmin);
        if (lane == 0 && tstar != 0u)
          __hip_atomic_fetch_max(row_thr(row_block(p, out_row(p, cur.rd))), tstar, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();
    }
    if (nxt.phase != 2) issue_tile<T>(p, nxt, nbuf, nthr, lane_off);
  } else {
    if (nxt.phase != 2) issue_tile<T>(p, nxt, nbuf, nthr, lane_off);
    process_tile<T, false>(p, cur, buf, thr, lane, s);
  }
}

// One worker wave.  Two tile buffers: while one tile is processed the next is in flight.
// A tile's record is stored while it is processed and the tile is counted at the top of
// the next step, after the wait that brings in the next tile (which also completes the
// record's stores).
template <typename T>
__device__ __forceinline__ void stream_worker(const StepArgs& p, WaveLds& s, uint64_t* pool, int g, int w,
                                              int lane) {
  const int rows = p.B * p.gamma;
  Task cur = task_at(g, rows, p.S, p.nt - p.S);
  uniform(cur);
  if (cur.phase == 2) return;
  const uint32_t lane_off = static_cast<uint32_t>(lane * Traits<T>::kPer * sizeof(T));
  u32x4 bufA[kSubGroups], bufB[kSubGroups];
  uint32_t thrA = 0u, thrB = 0u;
  int prev = -1;  // tag of the tile processed in the previous step
  issue_tile<T>(p, cur, bufA, thrA, lane_off);
  for (;;) {
    Task nxt = cur;
    advance(nxt, p, rows);
    wait_all_memory();
    if (prev >= 0) count_done(p, prev, lane);
    step_tile<T>(p, cur, nxt, bufA, thrA, bufB, thrB, lane_off, lane, s, pool, w);
    prev = out_row(p, cur.rd);
    cur = nxt;
    if (cur.phase == 2) break;
    nxt = cur;
    advance(nxt, p, rows);
    wait_all_memory();
    count_done(p, prev, lane);
    step_tile<T>(p, cur, nxt, bufB, thrB, bufA, thrA, lane_off, lane, s, pool, w);
    prev = out_row(p, cur.rd);
    cur = nxt;
    if (cur.phase == 2) break;
  }
  wait_all_memory();
  count_done(p, prev, lane);
}

// ---- row merge (searcher waves) -------------------------------------------------------------
constexpr int kItemCap = 4 * kWave;  // record slots loaded per round trip

struct MergeLds {
  uint64_t list[kListCap];
  uint64_t top[kWave];
  uint32_t meta[kMaxStepTiles];  // per tile: exact entries | groups << 8 | re-read flag << 16
  uint32_t item[kItemCap];       // record slots to load: entry slot, or group slot | 1 << 31
};

// Keeps the min(n, K) best of list[0..n) in list[0..), sorted (order value desc).  The
// list is walked in chunks of 64 - K entries placed behind the K best so far; every
// entry of the window counts the entries above it, and those with fewer than K move to
// their rank.
__device__ __forceinline__ int list_topk(MergeLds& m, int n, int K, int lane) {
  uint64_t* win = m.top;
  int held = 0;
  for (int base = 0; base < n; base += kWave - K) {
    const int take = n - base < kWave - K ? n - base : kWave - K;
    if (lane < take) win[held + lane] = m.list[base + lane];
    __builtin_amdgcn_wave_barrier();
    const int cnt = held + take;
    const uint64_t mine = lane < cnt ? win[lane] : 0ull;
    const int r = lane < cnt ? count_above(win, cnt, mine) : kWave;
    __builtin_amdgcn_wave_barrier();
    if (r < K) win[r] = mine;
    __builtin_amdgcn_wave_barrier();
    held = cnt < K ? cnt : K;
  }
  if (lane < held) m.list[lane] = win[lane];
  __builtin_amdgcn_wave_barrier();
  return held;
}

// Appends up to EPG values per lane (bit j of keep: val[j]) to the list, cutting it to
// its K best first if they might not fit.
template <int E>
__device__ __forceinline__ void list_add(MergeLds& m, int& n, int K, int lane, uint32_t keep, const uint64_t (&val)[E]) {
  int total = 0;
#pragma unroll
  for (int j = 0; j < E; ++j) total += popc(ballot((keep >> j) & 1u));
  if (total == 0) return;
  if (n + total > kListCap) {
    __builtin_amdgcn_wave_barrier();
    n = list_topk(m, n, K, lane);
  }
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const bool k = (keep >> j) & 1u;
    const uint64_t mk = ballot(k);
    if (k) m.list[n + static_cast<int>(lanes_below(mk))] = val[j];
    n += popc(mk);
  }
}

// Spins until *p >= target; false if the wait ran out of time.
__device__ __forceinline__ bool wait_counter(const uint32_t* p, uint32_t target, uint64_t t0) {
  for (;;) {
    const uint32_t v = __builtin_amdgcn_readfirstlane(load_agent32(p));
    if (v >= target) return true;
    if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) return false;
    __builtin_amdgcn_s_sleep(4);
  }
}

// Merges output row orow once all its tiles are in: LSE, the sorted top K (to the
// outputs, and ids / logits to ids_out / logit_out), then resets the row's counters.
// Memory round trips are few: the headers and the sample candidates together, then the
// record slots that hold anything, kItemCap at a time.
template <typename T>
__device__ __forceinline__ bool merge_row(const StepArgs& p, int orow, int lane, MergeLds& m, int32_t* ids_out,
                                          float* logit_out, uint64_t t0) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * EPG;
  const int nt = p.nt, K = p.K;
  const int64_t V = p.V;
  const int log_k = K == 4 ? 2 : (K == 8 ? 3 : 4);
  char* blk = row_block(p, orow);
  const bool ok = wait_counter(row_done(blk), static_cast<uint32_t>(nt), t0);

  // LSE from the tiles' (max, sum) pairs, each lane folding its tiles online; the tiles'
  // record sizes go to LDS.
  const uint64_t* hdr = row_hdr(blk);
  // Every tile has counted, so the threshold word is final: a lower bound of the row's
  // K-th largest key.
  const uint32_t tstar = __builtin_amdgcn_readfirstlane(load_agent32(row_thr(blk)));
  float lm = neg_inf(), ls = 0.f;
  for (int j = lane; j < nt; j += kWave) {
    const uint64_t h0 = load_agent(&hdr[2 * j]);
    const uint64_t h1 = load_agent(&hdr[2 * j + 1]);
    const float tm = __uint_as_float(static_cast<uint32_t>(h0));
    const float ts = __uint_as_float(static_cast<uint32_t>(h0 >> 32));
    m.meta[j] = static_cast<uint32_t>(h1);
    if (tm != neg_inf()) {
      const float nm = fmaxf(lm, tm);
      ls = (lm == neg_inf() ? 0.f : ls * fast_exp2((lm - nm) * kLog2e)) + ts * fast_exp2((tm - nm) * kLog2e);
      lm = nm;
    }
  }
  const float M = wave_max(lm);
  const float tot = wave_sum(lm == neg_inf() ? 0.f : ls * fast_exp2((lm - M) * kLog2e));
  const float lse = (M == neg_inf()) ? neg_inf() : M + fast_log2(tot) * kLn2;
  __builtin_amdgcn_wave_barrier();

  // Every candidate at or above the final threshold: the tiles' exact entries and the
  // elements of their groups.  The slots that hold anything are listed (from the record
  // sizes in LDS) and loaded kItemCap at a time.
  const uint64_t* ent = row_ent(p, blk);
  const uint64_t* grp = row_grp(p, blk);
  const uint32_t* gpos = row_gpos(p, blk);
  int n = 0;
  const int n_ent_slots = nt * K, n_slots = n_ent_slots + nt * kTileGroups;
  int q0 = 0;
  while (q0 < n_slots) {
    // Collect up to kItemCap live slots starting at q0.
    int items = 0;
    while (q0 < n_slots && items + kWave <= kItemCap) {
      const int q = q0 + lane;
      bool live = false;
      uint32_t code = 0u;
      if (q < n_ent_slots) {
        live = (q & (K - 1)) < static_cast<int>(m.meta[q >> log_k] & 0xFFu);
        code = static_cast<uint32_t>(q);
      } else if (q < n_slots) {
        const int u = q - n_ent_slots;
        live = (u % kTileGroups) < static_cast<int>((m.meta[u / kTileGroups] >> 8) & 0xFFu);
        code = static_cast<uint32_t>(u) | 0x80000000u;
      }
      const uint64_t mk = ballot(live);
      if (live) m.item[items + static_cast<int>(lanes_below(mk))] = code;
      items += popc(mk);
      q0 += kWave;
    }
    __builtin_amdgcn_wave_barrier();
    // Load them all, then filter.
    constexpr int kPer = kItemCap / kWave;
    uint64_t e0[kPer], e1[kPer];
    uint32_t pos[kPer];
    bool isg[kPer], has[kPer];
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int it = r * kWave + lane;
      has[r] = it < items;
      const uint32_t code = has[r] ? m.item[it] : 0u;
      isg[r] = (code >> 31) != 0u;
      const uint32_t slot = code & 0x7FFFFFFFu;
      e0[r] = 0ull;
      e1[r] = 0ull;
      pos[r] = 0u;
      if (has[r]) {
        if (isg[r]) {
          e0[r] = load_agent(&grp[2 * slot]);
          e1[r] = load_agent(&grp[2 * slot + 1]);
          pos[r] = load_agent32(&gpos[slot]);
        } else {
          e0[r] = load_agent(&ent[slot]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const u32x4 d{static_cast<uint32_t>(e0[r]), static_cast<uint32_t>(e0[r] >> 32), static_cast<uint32_t>(e1[r]),
                    static_cast<uint32_t>(e1[r] >> 32)};
      uint64_t val[EPG];
      uint32_t keep = 0u;
#pragma unroll
      for (int jj = 0; jj < EPG; ++jj) {
        const uint32_t word = d[jj * 4 / EPG];
        const uint32_t bits = EPG == 8 ? (word >> (16 * (jj & 1))) & 0xFFFFu : word;
        const uint32_t id = pos[r] + static_cast<uint32_t>(jj);
        val[jj] = isg[r] ? cand_order(Traits<T>::key_bits(bits), id) : (jj == 0 ? e0[r] : 0ull);
        const bool ok_j = has[r] && (isg[r] ? static_cast<int64_t>(id) < V : jj == 0) &&
                          static_cast<uint32_t>(val[jj] >> 32) >= tstar;
        keep |= ok_j ? (1u << jj) : 0u;
      }
      list_add<EPG>(m, n, K, lane, keep, val);
    }
    __builtin_amdgcn_wave_barrier();
  }
  // Tiles with more groups at the top than a record holds are read again (rare: long
  // runs of equal logits).
  const int64_t bi = orow / p.gamma, ii = orow - bi * p.gamma;
  const T* rp = static_cast<const T*>(p.logits) + bi * p.stride_b + ii * p.stride_i;
  const __amdgpu_buffer_rsrc_t rsrc = row_resource(rp, static_cast<uint32_t>(V * static_cast<int64_t>(sizeof(T))));
  const uint32_t lane_off = static_cast<uint32_t>(lane * EPG * sizeof(T));
  for (int j0 = 0; j0 < nt; j0 += kWave) {
    uint64_t redo = ballot(j0 + lane < nt && ((m.meta[j0 + lane < nt ? j0 + lane : 0] >> 16) & 1u));
    while (redo) {
      const int tile = j0 + __builtin_ctzll(redo);
      redo &= redo - 1;
      u32x4 buf[kSubGroups];
      load_full<T>(buf, rsrc, tile * SUB, lane_off);
      if ((tile + 1) * SUB > V) mask_tail<T>(buf, tile * SUB, V, lane);
#pragma unroll
      for (int g = 0; g < kSubGroups; ++g) {
        uint64_t val[EPG];
        uint32_t keep = 0u;
        const int64_t base = tile * SUB + (g * kWave + lane) * EPG;
#pragma unroll
        for (int jj = 0; jj < EPG; ++jj) {
          const uint32_t word = buf[g][jj * 4 / EPG];
          const uint32_t bits = EPG == 8 ? (word >> (16 * (jj & 1))) & 0xFFFFu : word;
          const uint32_t k = Traits<T>::key_bits(bits);
          val[jj] = cand_order(k, static_cast<uint32_t>(base + jj));
          keep |= (base + jj < V && k >= tstar) ? (1u << jj) : 0u;
        }
        list_add<EPG>(m, n, K, lane, keep, val);
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
  const int nk = list_topk(m, n, K, lane);

  if (lane < nk) {
    const uint64_t v = m.list[lane];
    const uint32_t key = static_cast<uint32_t>(v >> 32);
    const int32_t id = static_cast<int32_t>(~static_cast<uint32_t>(v));
    const float x = Traits<T>::from_key(key);
    const int64_t o = static_cast<int64_t>(orow) * K + lane;
    p.cand_ids[o] = id;
    p.cand_logit[o] = x;
    if (p.cand_logprob) p.cand_logprob[o] = x - lse;
    ids_out[lane] = id;
    logit_out[lane] = x;
  }
  if (lane == 0) {
    if (p.lse) p.lse[orow] = lse;
    // Every task of the row has finished with these words: leave them zero.
    store_agent32(row_done(blk), 0u);
    store_agent32(row_thr(blk), 0u);
  }
  __builtin_amdgcn_wave_barrier();
  return ok;
}

// ---- searchers ------------------------------------------------------------------------------
struct SearcherLayout {
  FastLayout fast;
  uint32_t clogit, rready, merge, total;
};

__host__ __device__ inline SearcherLayout searcher_layout(int gamma, int K, int W) {
  SearcherLayout L{};
  L.fast = fast_layout(gamma, K, W);
  uint32_t p = L.fast.total;
  L.clogit = p;
  p += static_cast<uint32_t>((gamma * K * sizeof(float) + 15) & ~static_cast<size_t>(15));
  L.rready = p;
  p += static_cast<uint32_t>((gamma * sizeof(uint32_t) + 15) & ~static_cast<size_t>(15));
  L.merge = p;
  p += static_cast<uint32_t>(kMergeWaves * ((sizeof(MergeLds) + 15) & ~static_cast<size_t>(15)));
  L.total = p;
  return L;
}

template <typename T, int KT, int R>
__device__ __forceinline__ void searcher(const StepArgs& p, const TreeArgs& a, const SelectorArgs& s, uint64_t magic_w,
                         unsigned char* smem, int w, int lane) {
  const int b = static_cast<int>(blockIdx.x);
  const int gamma = a.gamma;
  const SearcherLayout L = searcher_layout(gamma, KT, a.W);
  const FastSmem sm = fast_smem(smem, L.fast);
  float* clogit = reinterpret_cast<float*>(smem + L.clogit);
  uint32_t* rready = reinterpret_cast<uint32_t*>(smem + L.rready);
  for (int e = static_cast<int>(threadIdx.x); e < gamma; e += static_cast<int>(blockDim.x)) {
    sm.ready[e] = 0u;
    rready[e] = 0u;
  }
  __syncthreads();
  if (w == 0) {
    fast_search<KT, R, true>(a, sm, b, lane, magic_w);
    return;
  }
  if (w > kMergeWaves) return;
  MergeLds& ml = *reinterpret_cast<MergeLds*>(smem + L.merge +
                                              (w - 1) * ((sizeof(MergeLds) + 15) & ~static_cast<size_t>(15)));
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  for (int i = w - 1; i < gamma; i += kMergeWaves) {
    const int orow = b * gamma + i;
    const bool ok = merge_row<T>(p, orow, lane, ml, sm.cids + i * KT, clogit + i * KT, t0);
    if (!ok && lane == 0) store_agent32(ws_err(p), 1u);
    publish_slab(rready, i);
    if (i > 0) wait_slab(rready, i - 1);
    const int64_t bi = static_cast<int64_t>(b) * gamma + i;
    float* slab = sm.slab + i * KT * KT;
    bigram_tile_bf16<1>(s.phi, s.psi, s.gate + bi * s.r, s.V, s.r, i, KT, a.anchor + b,
                        i > 0 ? sm.cids + (i - 1) * KT : sm.cids, sm.cids + i * KT, clogit + i * KT, s.sc.alpha[i],
                        s.sc.lambda[i], nullptr, slab, nullptr, lane);
    slab_row_max<KT>(sm.slab, sm.rmax, i * KT + lane, lane < KT ? i * KT + KT : 0, kWave);
    publish_slab(sm.ready, i);
    float* gq = s.logq + bi * KT * KT;
#pragma unroll
    for (int e = lane; e < KT * KT; e += kWave) gq[e] = slab[e];
  }
}

template <typename T, int KT, int R>
__global__ __launch_bounds__(kStepWaves* kWave, 4) void draft_step_kernel(StepArgs p, TreeArgs a, SelectorArgs s,
                                                                           uint64_t magic_w) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  if (static_cast<int>(blockIdx.x) < p.B) {
    searcher<T, KT, R>(p, a, s, magic_w, smem_raw, w, lane);
    return;
  }
  WaveLds& ws = reinterpret_cast<WaveLds*>(smem_raw)[w];
  uint64_t* pool = reinterpret_cast<uint64_t*>(smem_raw + kStepWaves * sizeof(WaveLds));
  stream_worker<T>(p, ws, pool, (static_cast<int>(blockIdx.x) - p.B) * kStepWaves + w, w, lane);
}

}  // namespace

// ---- host side ------------------------------------------------------------------------------
StepPlan step_plan(int B, int gamma, int64_t V, int K, int dtype) {
  StepPlan pl{};
  const int64_t sub = static_cast<int64_t>(kSubGroups) * kWave * (dtype == 1 ? 8 : 4);
  const size_t rows = static_cast<size_t>(B) * gamma;
  pl.nt = static_cast<int>((V + sub - 1) / sub);
  pl.S = pl.nt < kSampleTiles ? pl.nt : kSampleTiles;
  size_t off = 16 + static_cast<size_t>(pl.nt) * 2 * sizeof(uint64_t);
  pl.off_ent = off;
  off += static_cast<size_t>(pl.nt) * K * sizeof(uint64_t);
  pl.off_grp = off;
  off += static_cast<size_t>(pl.nt) * kTileGroups * 2 * sizeof(uint64_t);
  pl.off_gpos = off;
  off += static_cast<size_t>(pl.nt) * kTileGroups * sizeof(uint32_t);
  pl.row_bytes = (off + 255) & ~static_cast<size_t>(255);
  pl.bytes = kRowBlocks + rows * pl.row_bytes;
  return pl;
}

bool draft_step_fused(int dtype, bool aligned, int B, int gamma, int64_t V, int K, int feat_dtype, int W) {
  if (!aligned || feat_dtype != 1 || B > kMaxStepSequences) return false;
  if ((V * (dtype == 1 ? 2 : 4)) % 16 != 0) return false;
  if (!draft_tree_fused(feat_dtype, gamma, K, W)) return false;
  const StepPlan pl = step_plan(B, gamma, V, K, dtype);
  if (pl.nt > kMaxStepTiles) return false;
  return static_cast<int64_t>(B) * gamma * pl.nt < (static_cast<int64_t>(1) << 31);
}

hipError_t launch_draft_step(const void* logits, int dtype, int B, int gamma, int64_t V, int64_t stride_b,
                             int64_t stride_i, int K, int32_t* cand_ids, float* cand_logit, float* cand_logprob,
                             float* lse, const SelectorArgs& s, const TreeArgs& a, void* workspace,
                             hipStream_t stream) {
  const StepPlan pl = step_plan(B, gamma, V, K, dtype);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  // Two workgroups of eight waves fit on a compute unit; the searchers take B slots.
  int workers = 2 * cus - B;
  if (workers < cus) workers = cus;

  StepArgs p{};
  p.logits = logits;
  p.V = V;
  p.stride_b = stride_b;
  p.stride_i = stride_i;
  p.B = B;
  p.gamma = gamma;
  p.K = K;
  p.nt = pl.nt;
  p.S = pl.S;
  p.nw = workers * kStepWaves;
  p.step0_rd = p.nw / pl.S;
  p.step0_j = p.nw % pl.S;
  const int ns = pl.nt - pl.S;
  p.step1_rd = ns > 0 ? p.nw / ns : 0;
  p.step1_j = ns > 0 ? p.nw % ns : 0;
  p.magic_b = (0x100000000ull + B - 1) / B;
  p.cand_ids = cand_ids;
  p.cand_logit = cand_logit;
  p.cand_logprob = cand_logprob;
  p.lse = lse;
  p.ws = static_cast<char*>(workspace);
  p.row_bytes = static_cast<uint32_t>(pl.row_bytes);
  p.off_ent = static_cast<uint32_t>(pl.off_ent);
  p.off_grp = static_cast<uint32_t>(pl.off_grp);
  p.off_gpos = static_cast<uint32_t>(pl.off_gpos);

  const uint64_t magic_w = (0x100000000ull + a.W - 1) / a.W;
  const size_t worker_smem = kStepWaves * sizeof(WaveLds) + kStepWaves * 16 * sizeof(uint64_t);
  const size_t search_smem = searcher_layout(gamma, K, a.W).total;
  const size_t smem = worker_smem > search_smem ? worker_smem : search_smem;
  const dim3 grid(static_cast<unsigned>(B + workers)), block(kStepWaves * kWave);
  const int wk = a.W * K;
#define UBT_STEP_LAUNCH(TT, KK, RR)                                                                         \
  do {                                                                                                      \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&draft_step_kernel<TT, KK, RR>),               \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));          \
    hipLaunchKernelGGL((draft_step_kernel<TT, KK, RR>), grid, block, smem, stream, p, a, s, magic_w);      \
  } while (0)
#define UBT_STEP_ROWS(TT, KK)       \
  do {                              \
    if (wk <= 64)                   \
      UBT_STEP_LAUNCH(TT, KK, 1);   \
    else if (wk <= 128)             \
      UBT_STEP_LAUNCH(TT, KK, 2);   \
    else if (wk <= 256)             \
      UBT_STEP_LAUNCH(TT, KK, 4);   \
    else if (wk <= 384)             \
      UBT_STEP_LAUNCH(TT, KK, 6);   \
    else                            \
      UBT_STEP_LAUNCH(TT, KK, 8);   \
  } while (0)
#define UBT_STEP_K(TT)         \
  do {                         \
    if (K == 4)                \
      UBT_STEP_ROWS(TT, 4);    \
    else if (K == 8)           \
      UBT_STEP_ROWS(TT, 8);    \
    else                       \
      UBT_STEP_ROWS(TT, 16);   \
  } while (0)
  if (dtype == 1)
    UBT_STEP_K(uint16_t);
  else
    UBT_STEP_K(float);
#undef UBT_STEP_K
#undef UBT_STEP_ROWS
#undef UBT_STEP_LAUNCH
  return hipGetLastError();
}

}  // namespace ubt
