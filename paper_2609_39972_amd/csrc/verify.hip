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
// 384 query rows).  The query rows of a key/value head are (node, head-in-group) pairs,
// node-major, so grouped heads share every key/value block, and the whole tree of a head
// fits one group at the usual shapes (65 nodes x 4 heads = 260 rows): keys and values
// are then read from HBM once.  Each wave holds up to 3 tiles of 16 query rows, so every
// operand fragment read from LDS feeds up to 3 MFMAs.  Keys stream in blocks of 32
// through LDS, double-buffered, the next block's global loads in flight while the
// current one is used.  K is stored as it is; V is stored transposed (d-major), so both
// products read MFMA operands with plain LDS loads:
//   S^T = K Q^T     (v_mfma_f32_16x16x32_bf16, A = a K tile, B = 16 queries)
//   O^T += V^T P^T  (A = a V^T tile, B = P^T straight from the S^T accumulators)
// S^T puts the scores of one query in one lane column, 8 keys per lane, so P^T needs no
// shuffle: the k order of the second product is permuted to match (slot t of lane group
// g is key 4g + t for t < 4 and 16 + 4g + t - 4 after), and V^T is read in that order.
// The running maximum is raised only when a score exceeds it by more than 2^8 (weights
// then stay below 256, exact enough in fp32 and bf16), so the rescaling of the output
// accumulators is off the steady-state path.
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kAttnWaves = 8;
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kTilesPerWave = 3;
constexpr int kAttnRows = 16 * kAttnWaves * kTilesPerWave;  // query rows per workgroup (384)
constexpr int kKB = 32;                                      // keys per block
constexpr int kVtStride = 36;  // bf16 per V^T row: 32 keys + 4, so the transposing writes
                               // of one wave hit each bank at most twice
constexpr float kRescaleGap = 8.f;  // log2 units a score may exceed the running maximum

template <int D>
struct AttnLds {
  uint16_t k[2][kKB][D + 8];
  uint16_t vt[2][D][kVtStride];
};

typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));

__device__ __forceinline__ v8bf as_v8bf(v4u v) { return __builtin_bit_cast(v8bf, v); }

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
  int B, N, H, Hkv, g, R, groups;  // R = N * g query rows per key/value head, in groups of 384
  int64_t Pmax;
  float scale_log2;  // scale * log2(e)
  void* out;
  int out_f32;
  float* lse;
};

// The 16-byte chunks of one key/value block that thread t stages: K rows as they are
// (chunk = 8 consecutive d of one key) and V as pairs of keys at the same 8 d, so that
// the transposed write packs two keys per 32-bit LDS word.
template <int D>
struct Stage {
  static constexpr int kChunks = D / 8;                                  // chunks per key row
  static constexpr int kKPerThread = (kKB * kChunks + kAttnThreads - 1) / kAttnThreads;  // 1
  v4u k[kKPerThread];
  v4u v0, v1;
};

// Every load is issued unconditionally (clamped to a valid row, the value then dropped),
// so the number of loads in flight is the same on every path and the compiler waits for
// exactly the ones a value needs.
template <int D>
__device__ __forceinline__ void stage_load(const AttnArgs& p, Stage<D>& s, int b, int h, int blk, int npb, int P,
                                           int nn, int t) {
  constexpr int C = Stage<D>::kChunks;
  const bool tree = blk >= npb;
  const int base = tree ? (blk - npb) * kKB : blk * kKB;
  const int lim = tree ? nn : P;  // >= base + 1 for every block that exists
  const int64_t S = tree ? p.N : p.Pmax;
  const uint16_t* ks = tree ? p.kt : p.kc;
  const uint16_t* vs = tree ? p.vt : p.vc;
  const v4u zero = v4u{0u, 0u, 0u, 0u};
  auto row_ptr = [&](const uint16_t* src, int key, int c) {
    const int kk = min(key, lim - 1);
    return reinterpret_cast<const v4u*>(src + ((static_cast<int64_t>(b) * S + kk) * p.Hkv + h) * D + 8 * c);
  };
#pragma unroll
  for (int i = 0; i < Stage<D>::kKPerThread; ++i) {
    const int id = t + kAttnThreads * i;
    const int row = min(id / C, kKB - 1), c = id % C;
    const v4u v = *row_ptr(ks, base + row, c);
    s.k[i] = (id / C < kKB && base + row < lim) ? v : zero;
  }
  const int kp = t % 16, c = min(t / 16, C - 1);
  const int k0 = base + 2 * kp;
  const bool in = t / 16 < C;  // 16 key pairs x C chunks: the first 16 C threads
  const v4u a = *row_ptr(vs, k0, c), bb = *row_ptr(vs, k0 + 1, c);
  s.v0 = (in && k0 < lim) ? a : zero;
  s.v1 = (in && k0 + 1 < lim) ? bb : zero;
}

template <int D>
__device__ __forceinline__ void stage_store(AttnLds<D>& lds, int st, const Stage<D>& s, int t) {
  constexpr int C = Stage<D>::kChunks;
#pragma unroll
  for (int i = 0; i < Stage<D>::kKPerThread; ++i) {
    const int id = t + kAttnThreads * i;
    const int row = id / C, c = id % C;
    if (row < kKB) *reinterpret_cast<v4u*>(&lds.k[st][row][8 * c]) = s.k[i];
  }
  const int kp = t % 16, c = t / 16;
  if (c < C) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t a = (s.v0[e / 2] >> (16 * (e % 2))) & 0xFFFFu;
      const uint32_t bb = (s.v1[e / 2] >> (16 * (e % 2))) & 0xFFFFu;
      *reinterpret_cast<uint32_t*>(&lds.vt[st][8 * c + e][2 * kp]) = a | (bb << 16);
    }
  }
}

template <int D>
__global__ __launch_bounds__(kAttnThreads) void tree_attention_kernel(AttnArgs p) {
  constexpr int DS = D / 32;  // k steps of S^T
  constexpr int DT = D / 16;  // output tiles of O^T
  constexpr int TW = kTilesPerWave;
  __shared__ AttnLds<D> lds;

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
  const int lane = t % kWave;
  const int lr = lane & 15, kg = lane >> 4;

  const int P = min(max(p.prefix_len[b], 0), static_cast<int>(p.Pmax));
  const int nn = min(max(p.n_nodes[b], 0), p.N);
  const int npb = (P + kKB - 1) / kKB;
  const int nblk = npb + (nn + kKB - 1) / kKB;
  const int words = (p.N + 31) / 32;

  // Tile j of this wave holds query rows r0 + 16 (w + 8 j) + [0, 16); this lane is the
  // column lr of each.
  const int r0 = grp * kAttnRows;
  int ntile = 0;  // tiles of this wave with at least one row (wave-uniform)
#pragma unroll
  for (int j = 0; j < TW; ++j) ntile += (r0 + 16 * (w + kAttnWaves * j) < p.R) ? 1 : 0;
  int n_of[TW], head_of[TW];
  bool rin[TW], live[TW];
  v4u qf[TW][DS];
  const uint32_t* mrow[TW];
#pragma unroll
  for (int j = 0; j < TW; ++j) {
    const int r = r0 + 16 * (w + kAttnWaves * j) + lr;
    rin[j] = r < p.R;
    n_of[j] = rin[j] ? r / p.g : 0;
    head_of[j] = h * p.g + (rin[j] ? r % p.g : 0);
    live[j] = rin[j] && n_of[j] < nn;
    const uint16_t* qr = p.q + ((static_cast<int64_t>(b) * p.N + n_of[j]) * p.H + head_of[j]) * D;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const v4u v = *reinterpret_cast<const v4u*>(qr + 32 * s + 8 * kg);
      qf[j][s] = live[j] ? v : v4u{0u, 0u, 0u, 0u};
    }
    mrow[j] = p.mask + (static_cast<int64_t>(b) * p.N + n_of[j]) * words;
  }

  v4f o[TW][DT];
  float m_run[TW], l_part[TW];
#pragma unroll
  for (int j = 0; j < TW; ++j) {
#pragma unroll
    for (int i = 0; i < DT; ++i) o[j][i] = v4f{0.f, 0.f, 0.f, 0.f};
    m_run[j] = neg_inf();
    l_part[j] = 0.f;
  }
  const float c = p.scale_log2;

  Stage<D> sg;
  if (nblk > 0) {
    stage_load<D>(p, sg, b, h, 0, npb, P, nn, t);
    stage_store<D>(lds, 0, sg, t);
  }
  // Nothing is in flight when the loop starts: the first MFMA of each block then waits
  // for no global load, and the next block's loads stay in flight behind the compute.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int blk = 0; blk < nblk; ++blk) {
    const int st = blk & 1;
    // This block's mask words, then the next block's K/V (the last block loads itself
    // again, unused), all unconditional.
    const int tb = blk >= npb ? blk - npb : 0;
    uint32_t mw[TW];
#pragma unroll
    for (int j = 0; j < TW; ++j) mw[j] = mrow[j][tb];
    stage_load<D>(p, sg, b, h, blk + 1 < nblk ? blk + 1 : blk, npb, P, nn, t);

    // ---- S^T = K Q^T for 32 keys and each tile ----
    v4f s0[TW], s1[TW];
#pragma unroll
    for (int j = 0; j < TW; ++j) s0[j] = s1[j] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const v4u a0 = *reinterpret_cast<const v4u*>(&lds.k[st][lr][32 * s + 8 * kg]);
      const v4u a1 = *reinterpret_cast<const v4u*>(&lds.k[st][16 + lr][32 * s + 8 * kg]);
#pragma unroll
      for (int j = 0; j < TW; ++j) {
        if (j < ntile) {
          s0[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(a0), as_v8bf(qf[j][s]), s0[j], 0, 0, 0);
          s1[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(a1), as_v8bf(qf[j][s]), s1[j], 0, 0, 0);
        }
      }
    }

    // ---- softmax weights: which of the lane's 8 keys each query sees ----
    // Bit t of vis: key 4 kg + t (t < 4) or 16 + 4 kg + t - 4 (t >= 4) of this block.
    const bool full = blk < npb && (blk + 1) * kKB <= P;  // a context block wholly inside the prefix
    uint32_t vis[TW];
    if (full) {
#pragma unroll
      for (int j = 0; j < TW; ++j) vis[j] = live[j] ? 0xFFu : 0u;
    } else if (blk < npb) {
      const int left = P - blk * kKB;  // 1..31 keys of the block inside the prefix
      const uint32_t all = (1u << left) - 1u;
      const uint32_t v = ((all >> (4 * kg)) & 0xFu) | (((all >> (16 + 4 * kg)) & 0xFu) << 4);
#pragma unroll
      for (int j = 0; j < TW; ++j) vis[j] = live[j] ? v : 0u;
    } else {
      const int left = nn - tb * kKB;
      const uint32_t in = left >= 32 ? ~0u : ((1u << left) - 1u);
#pragma unroll
      for (int j = 0; j < TW; ++j) {
        const uint32_t bits = live[j] ? (mw[j] & in) : 0u;
        vis[j] = ((bits >> (4 * kg)) & 0xFu) | (((bits >> (16 + 4 * kg)) & 0xFu) << 4);
      }
    }
    // Fully visible blocks use the scores as they are; only partial blocks mask: the
    // maximum over visible scores, and a zero weight for each invisible key.
    bool grow = false;
    float mxs[TW];
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      float mx;
      if (full) {
        mx = fmaxf(fmaxf(fmaxf(s0[j][0], s0[j][1]), fmaxf(s0[j][2], s0[j][3])),
                   fmaxf(fmaxf(s1[j][0], s1[j][1]), fmaxf(s1[j][2], s1[j][3])));
      } else {
        mx = neg_inf();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          mx = ((vis[j] >> e) & 1u) ? fmaxf(mx, s0[j][e]) : mx;
          mx = ((vis[j] >> (4 + e)) & 1u) ? fmaxf(mx, s1[j][e]) : mx;
        }
      }
      mxs[j] = mx * c;
      grow = grow || (mxs[j] > m_run[j] + kRescaleGap);
    }
    if (ballot(grow)) {
      // Raise the running maxima that fell behind (uniform over each query's 4 lanes).
#pragma unroll
      for (int j = 0; j < TW; ++j) {
        float mx = mxs[j];
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        if (mx > m_run[j] + kRescaleGap) {
          const float alpha = __builtin_amdgcn_exp2f(m_run[j] - mx);
          m_run[j] = mx;
          l_part[j] *= alpha;
#pragma unroll
          for (int i = 0; i < DT; ++i) o[j][i] *= alpha;
        }
      }
    }
    v4u pt[TW];
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      // A stored row sees a visible key in its first block, so m_run is finite there; rows
      // never stored may turn NaN, which stays in their own column.
      const float nm = -m_run[j];
      float pr[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pr[e] = __builtin_amdgcn_exp2f(fmaf(s0[j][e], c, nm));
        pr[4 + e] = __builtin_amdgcn_exp2f(fmaf(s1[j][e], c, nm));
      }
      if (!full) {
#pragma unroll
        for (int e = 0; e < 8; ++e) pr[e] = ((vis[j] >> e) & 1u) ? pr[e] : 0.f;
      }
      l_part[j] += ((pr[0] + pr[1]) + (pr[2] + pr[3])) + ((pr[4] + pr[5]) + (pr[6] + pr[7]));
      pt[j] = v4u{pack_bf16(pr[0], pr[1]), pack_bf16(pr[2], pr[3]), pack_bf16(pr[4], pr[5]),
                  pack_bf16(pr[6], pr[7])};
    }

    // ---- O^T += V^T P^T ----
#pragma unroll
    for (int i = 0; i < DT; ++i) {
      const uint16_t* vrow = &lds.vt[st][16 * i + lr][0];
      const v2u lo = *reinterpret_cast<const v2u*>(vrow + 4 * kg);
      const v2u hi = *reinterpret_cast<const v2u*>(vrow + 16 + 4 * kg);
      const v4u a = v4u{lo.x, lo.y, hi.x, hi.y};
#pragma unroll
      for (int j = 0; j < TW; ++j)
        if (j < ntile) o[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(a), as_v8bf(pt[j]), o[j][i], 0, 0, 0);
    }

    if (blk + 1 < nblk) stage_store<D>(lds, st ^ 1, sg, t);
    __syncthreads();
  }

  // ---- normalise and store: lane (lr, kg) holds d = 16 i + 4 kg + e of its query ----
#pragma unroll
  for (int j = 0; j < TW; ++j) {
    float l = l_part[j] + __shfl_xor(l_part[j], 16);
    l = l + __shfl_xor(l, 32);
    if (!rin[j]) continue;
    const bool has = live[j] && l > 0.f;
    const float inv = has ? 1.f / l : 0.f;
    const int64_t orow = (static_cast<int64_t>(b) * p.N + n_of[j]) * p.H + head_of[j];
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
    if (p.lse && kg == 0) p.lse[orow] = has ? (m_run[j] + __builtin_amdgcn_logf(l)) * kLn2 : neg_inf();
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
  if (a.D == 128)
    hipLaunchKernelGGL(tree_attention_kernel<128>, grid, dim3(kAttnThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(tree_attention_kernel<64>, grid, dim3(kAttnThreads), 0, stream, p);
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
