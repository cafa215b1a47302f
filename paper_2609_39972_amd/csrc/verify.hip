// Verification of a draft tree: tree attention, the acceptance walk and the KV commit.
//
// Appendix A / Verification via Tree-attention: the prefix-closed tree is verified in
// one target forward pass in which every node is evaluated under its own prefix (the
// committed context, then its ancestors and itself: the ancestor mask); the walk
// follows the child that matches the target's sample until the first mismatch, whose
// sample is the bonus token; the key/value rows along the accepted path are carried
// into the cache and the other branches are dropped.  Background, "Tree Drafting".
//
// Tree attention: one workgroup of 4 waves per (sequence, key/value head, 64 query
// rows).  The query rows of a key/value head are (node, head-in-group) pairs, node-major,
// so grouped heads share every key/value block.  Keys stream in blocks of 32 through
// LDS, double-buffered, the next block's global loads in flight while the current one is
// used.  K is stored as it is; V is stored transposed (d-major), so both products read
// MFMA operands with plain LDS loads:
//   S^T = K Q^T     (v_mfma_f32_16x16x32_bf16, A = a K tile, B = the wave's 16 queries)
//   O^T += V^T P^T  (A = a V^T tile, B = P^T straight from the S^T accumulators)
// S^T puts the scores of one query in one lane column, 8 keys per lane, so the online
// softmax reduces over two cross-lane steps and P^T needs no shuffle: the k order of the
// second product is permuted to match (slot t of lane group g is key 4g + t for t < 4
// and 16 + 4g + t - 4 after), and the V^T operand is read in the same order.
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kAttnWaves = 4;
constexpr int kAttnRows = 16 * kAttnWaves;  // query rows per workgroup
constexpr int kKB = 32;                      // keys per block
constexpr int kVtStride = 36;  // bf16 per V^T row: 32 keys + 4, so the transposing writes
                               // of one wave hit each bank at most twice

template <int D>
struct AttnLds {
  uint16_t k[2][kKB][D + 8];
  uint16_t vt[2][D][kVtStride];
};

__device__ __forceinline__ v8bf as_v8bf(v4u v) { return __builtin_bit_cast(v8bf, v); }

// Round-to-nearest-even to bf16 of a finite non-negative float (the probabilities).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) { return bf16_rne(lo) | (bf16_rne(hi) << 16); }

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* prefix_len;
  const uint16_t* kt;
  const uint16_t* vt;
  const uint32_t* mask;
  const int32_t* n_nodes;
  int B, N, H, Hkv, g, R, tiles;  // R = N * g query rows per key/value head; tiles = ceil(R / 64)
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
  static constexpr int kKPerThread = (kKB * kChunks + 255) / 256;        // 2 (D = 128) or 1 (D = 64)
  v4u k[kKPerThread];
  v4u v0, v1;
};

template <int D>
__device__ __forceinline__ void stage_load(const AttnArgs& p, Stage<D>& s, int b, int h, int blk, int npb, int P,
                                           int nn, int t) {
  constexpr int C = Stage<D>::kChunks;
  const bool tree = blk >= npb;
  const int base = tree ? (blk - npb) * kKB : blk * kKB;
  const int lim = tree ? nn : P;
  const int64_t S = tree ? p.N : p.Pmax;
  const uint16_t* ks = tree ? p.kt : p.kc;
  const uint16_t* vs = tree ? p.vt : p.vc;
  const v4u zero = v4u{0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < Stage<D>::kKPerThread; ++i) {
    const int id = t + 256 * i;
    const int row = id / C, c = id % C;
    const int key = base + row;
    s.k[i] = (row < kKB && key < lim)
                 ? *reinterpret_cast<const v4u*>(ks + ((static_cast<int64_t>(b) * S + key) * p.Hkv + h) * D + 8 * c)
                 : zero;
  }
  const int kp = t % 16, c = t / 16;
  const int k0 = base + 2 * kp;
  const bool in = c < C;
  s.v0 = (in && k0 < lim) ? *reinterpret_cast<const v4u*>(vs + ((static_cast<int64_t>(b) * S + k0) * p.Hkv + h) * D + 8 * c)
                          : zero;
  s.v1 = (in && k0 + 1 < lim)
             ? *reinterpret_cast<const v4u*>(vs + ((static_cast<int64_t>(b) * S + k0 + 1) * p.Hkv + h) * D + 8 * c)
             : zero;
}

template <int D>
__device__ __forceinline__ void stage_store(AttnLds<D>& lds, int st, const Stage<D>& s, int t) {
  constexpr int C = Stage<D>::kChunks;
#pragma unroll
  for (int i = 0; i < Stage<D>::kKPerThread; ++i) {
    const int id = t + 256 * i;
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
__global__ __launch_bounds__(256) void tree_attention_kernel(AttnArgs p) {
  constexpr int DS = D / 32;  // k steps of S^T
  constexpr int DT = D / 16;  // output tiles of O^T
  __shared__ AttnLds<D> lds;

  // Workgroup -> (sequence, key/value head, row tile).  Consecutive workgroups go to
  // different XCDs; the remap puts the row tiles of one (sequence, head) on one XCD, so
  // their key/value blocks are shared through that XCD's L2.
  const int total = p.B * p.Hkv * p.tiles;
  const int L = static_cast<int>(blockIdx.x);
  const int T8 = total - total % 8;
  const int id = L < T8 ? (L % 8) * (T8 / 8) + L / 8 : L;
  const int tile = id % p.tiles;
  const int bh = id / p.tiles;
  const int h = bh % p.Hkv;
  const int b = bh / p.Hkv;

  const int t = static_cast<int>(threadIdx.x);
  const int w = t / kWave, lane = t % kWave;
  const int lr = lane & 15, kg = lane >> 4;

  const int P = min(max(p.prefix_len[b], 0), static_cast<int>(p.Pmax));
  const int nn = min(max(p.n_nodes[b], 0), p.N);
  const int npb = (P + kKB - 1) / kKB;
  const int nblk = npb + (nn + kKB - 1) / kKB;
  const int words = (p.N + 31) / 32;

  // This lane's query row (B operand column and softmax column).
  const int r = tile * kAttnRows + w * 16 + lr;
  const bool rin = r < p.R;
  const int n = rin ? r / p.g : 0;
  const int head = h * p.g + (rin ? r % p.g : 0);
  const bool live = rin && n < nn;
  v4u qf[DS];
  {
    const uint16_t* qr = p.q + ((static_cast<int64_t>(b) * p.N + n) * p.H + head) * D;
#pragma unroll
    for (int s = 0; s < DS; ++s)
      qf[s] = live ? *reinterpret_cast<const v4u*>(qr + 32 * s + 8 * kg) : v4u{0u, 0u, 0u, 0u};
  }
  const uint32_t* mrow = p.mask + (static_cast<int64_t>(b) * p.N + n) * words;

  v4f o[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i) o[i] = v4f{0.f, 0.f, 0.f, 0.f};
  float m_run = neg_inf(), l_part = 0.f;

  Stage<D> sg;
  if (nblk > 0) {
    stage_load<D>(p, sg, b, h, 0, npb, P, nn, t);
    stage_store<D>(lds, 0, sg, t);
  }
  __syncthreads();
  for (int blk = 0; blk < nblk; ++blk) {
    const int st = blk & 1;
    if (blk + 1 < nblk) stage_load<D>(p, sg, b, h, blk + 1, npb, P, nn, t);

    // ---- S^T = K Q^T for 32 keys ----
    v4f s0 = v4f{0.f, 0.f, 0.f, 0.f}, s1 = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const v4u a0 = *reinterpret_cast<const v4u*>(&lds.k[st][lr][32 * s + 8 * kg]);
      const v4u a1 = *reinterpret_cast<const v4u*>(&lds.k[st][16 + lr][32 * s + 8 * kg]);
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(a0), as_v8bf(qf[s]), s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(a1), as_v8bf(qf[s]), s1, 0, 0, 0);
    }

    // ---- which of the lane's 8 keys this query sees ----
    // bit t of vis: key 4 kg + t (t < 4) or 16 + 4 kg + t - 4 (t >= 4) of this block.
    uint32_t vis;
    if (blk < npb) {
      const int left = P - blk * kKB;  // keys of the block inside the prefix
      uint32_t all = left >= 32 ? ~0u : ((1u << left) - 1u);
      vis = ((all >> (4 * kg)) & 0xFu) | (((all >> (16 + 4 * kg)) & 0xFu) << 4);
    } else {
      const int tb = blk - npb;
      const int left = nn - tb * kKB;
      const uint32_t in = left >= 32 ? ~0u : ((1u << left) - 1u);
      const uint32_t bits = live ? (mrow[tb] & in) : 0u;
      vis = ((bits >> (4 * kg)) & 0xFu) | (((bits >> (16 + 4 * kg)) & 0xFu) << 4);
    }
    if (!live) vis = 0u;
    float x[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = ((vis >> j) & 1u) ? s0[j] * p.scale_log2 : neg_inf();
      x[4 + j] = ((vis >> (4 + j)) & 1u) ? s1[j] * p.scale_log2 : neg_inf();
    }
    float mb = x[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) mb = fmaxf(mb, x[j]);
    mb = fmaxf(mb, __shfl_xor(mb, 16));
    mb = fmaxf(mb, __shfl_xor(mb, 32));
    const float m_new = fmaxf(m_run, mb);
    const bool any = m_new != neg_inf();
    const float alpha = any ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.f;
    float pr[8];
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      pr[j] = ((vis >> j) & 1u) ? __builtin_amdgcn_exp2f(x[j] - m_new) : 0.f;
      psum += pr[j];
    }
    l_part = l_part * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < DT; ++i) o[i] *= alpha;
    const v4u pt = v4u{pack_bf16(pr[0], pr[1]), pack_bf16(pr[2], pr[3]), pack_bf16(pr[4], pr[5]),
                       pack_bf16(pr[6], pr[7])};

    // ---- O^T += V^T P^T ----
#pragma unroll
    for (int i = 0; i < DT; ++i) {
      const uint16_t* vrow = &lds.vt[st][16 * i + lr][0];
      const v2u lo = *reinterpret_cast<const v2u*>(vrow + 4 * kg);
      const v2u hi = *reinterpret_cast<const v2u*>(vrow + 16 + 4 * kg);
      const v4u a = v4u{lo.x, lo.y, hi.x, hi.y};
      o[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_v8bf(a), as_v8bf(pt), o[i], 0, 0, 0);
    }

    if (blk + 1 < nblk) stage_store<D>(lds, st ^ 1, sg, t);
    __syncthreads();
  }

  // ---- normalise and store: lane (lr, kg) holds d = 16 i + 4 kg + j of its query ----
  float l = l_part + __shfl_xor(l_part, 16);
  l = l + __shfl_xor(l, 32);
  if (!rin) return;
  const bool has = live && l > 0.f;
  const float inv = has ? 1.f / l : 0.f;
  const int64_t orow = (static_cast<int64_t>(b) * p.N + n) * p.H + head;
  if (p.out_f32) {
    float* op = static_cast<float*>(p.out) + orow * D;
#pragma unroll
    for (int i = 0; i < DT; ++i) *reinterpret_cast<v4f*>(op + 16 * i + 4 * kg) = o[i] * inv;
  } else {
    uint16_t* op = static_cast<uint16_t*>(p.out) + orow * D;
#pragma unroll
    for (int i = 0; i < DT; ++i) {
      const v4f v = o[i] * inv;
      // The output rounds to nearest even like the probabilities, here with sign.
      uint32_t e[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t u = __float_as_uint(v[j]);
        e[j] = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
      }
      *reinterpret_cast<v2u*>(op + 16 * i + 4 * kg) = v2u{e[0] | (e[1] << 16), e[2] | (e[3] << 16)};
    }
  }
  if (p.lse && kg == 0) p.lse[orow] = has ? (m_run + __builtin_amdgcn_logf(l)) * kLn2 : neg_inf();
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
  p.tiles = (p.R + kAttnRows - 1) / kAttnRows;
  p.Pmax = a.Pmax;
  p.scale_log2 = a.scale * kLog2e;
  p.out = a.out;
  p.out_f32 = a.out_f32;
  p.lse = a.lse;
  const dim3 grid(static_cast<unsigned>(p.B * p.Hkv * p.tiles));
  if (a.D == 128)
    hipLaunchKernelGGL(tree_attention_kernel<128>, grid, dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL(tree_attention_kernel<64>, grid, dim3(256), 0, stream, p);
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
