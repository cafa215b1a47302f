// Best-first tree under the unigram-plus-bigram scoring.
//
// Each edge scores its successor's unigram log-probability (Method / Unigram Proposer,
// Eq. ubtree-unigram) plus the raw selector score (Background, Eq. dflash2-selector),
// weighted as in Method / Depth Calibration, Eq. (ubtree-depth), without normalising over
// the successors; a path scores the cumulative sum of its edges plus zeta per depth
// (Appendix A, Eq. ubtree-depth-bonus).  Paths are grown best-first (Background, "Tree
// Drafting"): from the root, the best node among the children of the tree's nodes joins
// the tree, until `budget` nodes are in.  These sums can rise along a path, so the prefix
// closure that Appendix A / Global Pruning obtains from normalised scores comes from the
// growth rule itself: a node becomes eligible only once its parent is in the tree.
//
// Order among eligible nodes: score desc, then depth asc, then the parent's slot asc,
// then the candidate rank asc.  Slots are assigned in growth order (root = 0).
//
// One wavefront per sequence; everything in registers and LDS.  The eligible set is
// never materialised: when a node joins the tree its K children's scores are formed and
// ranked once (score desc, rank asc), and the node keeps a cursor on that list, so its
// best remaining child is its "head".  Every eligible node is a head or a sibling behind
// a head, so the best eligible node is the best head: one 64-bit wave maximum per step.
// Lane l holds the heads and cursors of slots l, l + 64, l + 128 and l + 192.
#include "search.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

// Edge slabs stay in LDS up to this size (the whole layout then stays under 64 KB);
// larger ones (K = 64, or K = 16 beyond 32 positions) are read from memory.
constexpr size_t kBfSlabLdsBytes = 32 * 1024;

struct BfLayout {
  uint32_t slab, order, nscore, ninfo, csum, anc, mk, total;
};

__host__ __device__ inline BfLayout bf_layout(int gamma, int K, int N, bool slab_lds) {
  BfLayout L{};
  uint32_t p = 0;
  auto take = [&p](size_t bytes) {
    const uint32_t at = p;
    p += static_cast<uint32_t>((bytes + 15) & ~static_cast<size_t>(15));
    return at;
  };
  L.slab = take(slab_lds ? static_cast<size_t>(gamma) * K * K * sizeof(float) : 0);
  L.order = take(static_cast<size_t>(N) * K);  // per slot: its children's ranks in score order
  L.nscore = take(static_cast<size_t>(N) * sizeof(float));
  L.ninfo = take(static_cast<size_t>(N) * sizeof(uint32_t));
  L.csum = take(kWave * sizeof(float));
  L.anc = take(kMaxNodes * sizeof(int32_t));
  L.mk = take(kMaxNodes * kMaskWords * sizeof(uint32_t));
  L.total = p;
  return L;
}

// Slot info: depth (bits 0-7), candidate rank (bits 8-15), parent slot + 1 (bits 16-24).
__device__ __forceinline__ uint32_t pack_info(int d, int c, int p) {
  return static_cast<uint32_t>(d) | (static_cast<uint32_t>(c) << 8) | (static_cast<uint32_t>(p + 1) << 16);
}

// Head value of slot p's child at depth d with score v: larger is better under (score
// desc, depth asc, parent slot asc).  Never 0 (f32_key of a non-NaN value is nonzero).
__device__ __forceinline__ uint64_t head_value(float v, int d, int p) {
  return (static_cast<uint64_t>(f32_key(v)) << 32) | ~((static_cast<uint32_t>(d) << 8) | static_cast<uint32_t>(p));
}

template <bool kSlabLds>
__global__ __launch_bounds__(kWave) void best_first_kernel(TreeArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int lane = static_cast<int>(threadIdx.x);
  const int64_t b = blockIdx.x;
  const int gamma = a.gamma, K = a.K, budget = a.budget, N = budget + 1;
  const BfLayout L = bf_layout(gamma, K, N, kSlabLds);
  const int slab_n = gamma * K * K;
  const float* gslab = a.logq + b * slab_n;
  float* lslab = reinterpret_cast<float*>(smem_raw + L.slab);
  if (kSlabLds) {
    if ((reinterpret_cast<uintptr_t>(gslab) & 15u) == 0 && (slab_n & 3) == 0) {
      const float4* src = reinterpret_cast<const float4*>(gslab);
      float4* dst = reinterpret_cast<float4*>(lslab);
      for (int e = lane; e < slab_n / 4; e += kWave) dst[e] = src[e];
    } else {
      for (int e = lane; e < slab_n; e += kWave) lslab[e] = gslab[e];
    }
  }
  const float* E = kSlabLds ? lslab : gslab;
  unsigned char* order = smem_raw + L.order;
  float* nscore = reinterpret_cast<float*>(smem_raw + L.nscore);
  uint32_t* ninfo = reinterpret_cast<uint32_t*>(smem_raw + L.ninfo);
  float* csum = reinterpret_cast<float*>(smem_raw + L.csum);
  int32_t* anc = reinterpret_cast<int32_t*>(smem_raw + L.anc);
  uint32_t* mk = reinterpret_cast<uint32_t*>(smem_raw + L.mk);
  const float zeta = a.zeta;
  const bool with_zeta = zeta != 0.f;
  __syncthreads();

  uint64_t hv[4] = {0ull, 0ull, 0ull, 0ull};  // heads of slots lane + 64 j (0: none)
  int cur[4] = {0, 0, 0, 0};                  // cursors into those slots' child lists

  // Slot s (depth d, candidate rank c, score sc) has joined the tree: rank its children
  // (score desc, rank asc) into order[s], and set its head.
  auto expand = [&](int s, int d, int c, float sc) {
    if (d >= gamma) return;  // wave-uniform: no children past the last position
    const float* row = E + (static_cast<int64_t>(d) * K + (d == 0 ? 0 : c)) * K;
    float v = 0.f;
    if (lane < K) {
      v = sc + row[lane];
      if (with_zeta) v += zeta;
      csum[lane] = v;
    }
    __builtin_amdgcn_wave_barrier();
    int rank = 0;
    if (lane < K) {
      for (int j = 0; j < K; ++j) {
        const float x = csum[j];
        rank += (x > v || (x == v && j < lane)) ? 1 : 0;
      }
      order[s * K + rank] = static_cast<unsigned char>(lane);
    }
    const uint64_t first = ballot(lane < K && rank == 0);
    const int fl = __builtin_ctzll(first);
    const float best = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), fl));
    const uint64_t h = head_value(best, d + 1, s);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lane == (s & 63) && j == (s >> 6)) {
        hv[j] = h;
        cur[j] = 0;
      }
    __builtin_amdgcn_wave_barrier();
  };

  if (lane == 0) {
    nscore[0] = 0.f;
    ninfo[0] = pack_info(0, 0, -1);
  }
  expand(0, 0, 0, 0.f);
  int n = 1;
  for (; n <= budget; ++n) {
    // The best head: the largest score key, then among those the largest low word.
    uint32_t hi = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) hi = max(hi, static_cast<uint32_t>(hv[j] >> 32));
    const uint32_t hmax = wave_umax(hi);
    if (hmax == 0u) break;  // wave-uniform: nothing left to grow
    uint32_t lo = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (static_cast<uint32_t>(hv[j] >> 32) == hmax) lo = max(lo, static_cast<uint32_t>(hv[j]));
    const uint32_t dp = ~wave_umax(lo);
    const int d = static_cast<int>(dp >> 8);     // the new node's depth
    const int p = static_cast<int>(dp & 0xFFu);  // its parent's slot
    const float sc = f32_key_value(hmax);
    // The parent's cursor names the new node's candidate rank.
    int cp = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j == (p >> 6)) cp = __builtin_amdgcn_readlane(cur[j], p & 63);
    const int c = order[p * K + cp];
    if (lane == 0) {
      nscore[n] = sc;
      ninfo[n] = pack_info(d, c, p);
    }
    // The parent's next child becomes its head.
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lane == (p & 63) && j == (p >> 6)) {
        const int nc = cur[j] + 1;
        cur[j] = nc;
        uint64_t h = 0ull;
        if (nc < K) {
          const int c2 = order[p * K + nc];
          const uint32_t pinfo = ninfo[p];
          const int pc = static_cast<int>((pinfo >> 8) & 0xFFu);
          const float* row = E + (static_cast<int64_t>(d - 1) * K + (d == 1 ? 0 : pc)) * K;
          float v2 = nscore[p] + row[c2];
          if (with_zeta) v2 += zeta;
          h = head_value(v2, d, p);
        }
        hv[j] = h;
      }
    expand(n, d, c, sc);
  }
  const int n_nodes = n;

  // ---- outputs -------------------------------------------------------------------------
  const int words = (N + 31) / 32;
  int32_t* tok = a.token + b * N;
  int32_t* par = a.parent + b * N;
  int32_t* dep = a.depth + b * N;
  int32_t* crk = a.cand_rank + b * N;
  float* scr = a.score + b * N;
  if (lane == 0) a.n_nodes[b] = n_nodes;
  for (int t = lane; t < N; t += kWave) {
    if (t < n_nodes) {
      const uint32_t info = ninfo[t];
      const int d = static_cast<int>(info & 0xFFu);
      const int c = static_cast<int>((info >> 8) & 0xFFu);
      const int p = static_cast<int>(info >> 16) - 1;
      tok[t] = t == 0 ? a.anchor[b] : a.cand_ids[(b * gamma + d - 1) * K + c];
      par[t] = p;
      dep[t] = d;
      crk[t] = t == 0 ? -1 : c;
      scr[t] = nscore[t];
      anc[t] = p;
    } else {
      tok[t] = -1;
      par[t] = -1;
      dep[t] = -1;
      crk[t] = -1;
      scr[t] = neg_inf();
    }
  }
  __builtin_amdgcn_wave_barrier();
  if (a.mask) {
    const int max_depth = gamma < budget ? gamma : budget;
    ancestor_mask(anc, mk, n_nodes, N, max_depth, a.mask + b * static_cast<int64_t>(N) * words, lane);
  }
}

}  // namespace

hipError_t launch_best_first(const TreeArgs& a, hipStream_t stream) {
  const int N = a.budget + 1;
  const bool slab_lds = static_cast<size_t>(a.gamma) * a.K * a.K * sizeof(float) <= kBfSlabLdsBytes;
  const size_t smem = bf_layout(a.gamma, a.K, N, slab_lds).total;
  const dim3 grid(static_cast<unsigned>(a.B)), block(kWave);
  if (slab_lds) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&best_first_kernel<true>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    hipLaunchKernelGGL((best_first_kernel<true>), grid, block, smem, stream, a);
  } else {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&best_first_kernel<false>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    hipLaunchKernelGGL((best_first_kernel<false>), grid, block, smem, stream, a);
  }
  return hipGetLastError();
}

}  // namespace ubt
