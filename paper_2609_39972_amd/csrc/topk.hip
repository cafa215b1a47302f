// Softmax statistics and top-K candidate selection over the full vocabulary.
//
// Method / Unigram Proposer, Eq. (ubtree-unigram), q_i = softmax(u_i), and "Candidate
// Sets": C_i = the K tokens of largest q_i, ranked here on the logits (softmax is
// increasing) with ties to the lower token id.
//
// One HBM pass.  A row of V logits is cut into P chunks of 64 lanes x 16 groups x 16 B
// (8192 bf16 or 4096 fp32 elements); each wavefront owns one chunk and keeps it in
// registers.  Per 16-byte group it takes the group maximum and the exp-sum relative to
// it, folds both into a running per-lane (max, sum), and remembers the group maximum.
// The K-th largest lane maximum tau bounds the chunk's K-th largest element from below,
// so only groups whose maximum reaches tau can hold a top-K element; those few groups
// go to LDS, and a ballot-driven radix selection picks the chunk's top K.  Every wave
// writes (max, sum) and its K candidates to the workspace; the last wave of a row to
// finish (atomic counter) merges the P partials into the row's LSE and sorted top-K.
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

constexpr int kGroups = 16;         // 16-byte groups per lane per chunk
constexpr int kWavesPerBlock = 4;   // independent waves per workgroup
constexpr int kCapGroups = 32;      // LDS candidate-group buffer per wave and round

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T>
struct Traits;

template <>
struct Traits<uint16_t> {  // bf16 bit patterns
  static constexpr int kPer = 8;
  static constexpr int kKeyBits = 16;
    __device__ static float elem(const u32x4& v, int j) {
    const uint32_t w = v[j >> 1];
    return __uint_as_float((j & 1) ? (w & 0xFFFF0000u) : (w << 16));
  }
  __device__ static uint32_t elem_bits(const u32x4& v, int j) { return (v[j >> 1] >> (16 * (j & 1))) & 0xFFFFu; }
  __device__ static uint32_t key_bits(uint32_t bits) { return bf16_key(bits); }
  __device__ static uint32_t key_value(float f) { return bf16_key(__float_as_uint(f) >> 16); }
  __device__ static float from_key(uint32_t k) { return bf16_key_value(k); }
  __device__ static void set_neg_inf(u32x4& v) { v = u32x4{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u}; }
  __device__ static void set_elem(u32x4& v, int j, uint32_t bits) {
    const int s = 16 * (j & 1);
    v[j >> 1] = (v[j >> 1] & ~(0xFFFFu << s)) | (bits << s);
  }
  __device__ static uint32_t load_elem(const uint16_t* p) { return *p; }
};

template <>
struct Traits<float> {
  static constexpr int kPer = 4;
  static constexpr int kKeyBits = 32;
  __device__ static float elem(const u32x4& v, int j) { return __uint_as_float(v[j]); }
  __device__ static uint32_t elem_bits(const u32x4& v, int j) { return v[j]; }
  __device__ static uint32_t key_bits(uint32_t bits) { return f32_key(__uint_as_float(bits)); }
  __device__ static uint32_t key_value(float f) { return f32_key(f); }
  __device__ static float from_key(uint32_t k) { return f32_key_value(k); }
  __device__ static void set_neg_inf(u32x4& v) { v = u32x4{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u}; }
  __device__ static void set_elem(u32x4& v, int j, uint32_t bits) { v[j] = bits; }
  __device__ static uint32_t load_elem(const float* p) { return __float_as_uint(*p); }
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Stores and loads that are coherent at device (agent) scope: partial results travel
// between waves on different XCDs without cache-wide writeback or invalidation.
__device__ __forceinline__ void store_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_agent(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t pack(uint32_t lo, uint32_t hi) {
  return static_cast<uint64_t>(lo) | (static_cast<uint64_t>(hi) << 32);
}

// Group of EPG elements starting at element e0 of row `rp`, elements >= lim read as -inf.
template <typename T, bool kAligned>
__device__ __forceinline__ u32x4 load_group_checked(const T* rp, int64_t e0, int64_t lim) {
  constexpr int EPG = Traits<T>::kPer;
  u32x4 v;
  if (kAligned && e0 + EPG <= lim) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(rp + e0));
  Traits<T>::set_neg_inf(v);
#pragma unroll
  for (int j = 0; j < EPG; ++j)
    if (e0 + j < lim) Traits<T>::set_elem(v, j, Traits<T>::load_elem(rp + e0 + j));
  return v;
}

struct WaveLds {
  u32x4 data[kCapGroups];      // buffered candidate groups
  uint32_t base[kCapGroups];   // chunk-relative index of each group's first element
  uint2 stage[kWave];          // compaction staging (key, id)
};

// Compacts the selected entries (at most 64) into lanes 0.. of (out_key, out_id).
template <int R>
__device__ __forceinline__ int compact(WaveLds& s, const uint32_t (&key)[R], const uint32_t (&sub)[R],
                                       const uint64_t (&sel)[R], int lane, uint32_t& out_key, uint32_t& out_id) {
  int n = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if ((sel[r] >> lane) & 1ull) s.stage[n + lanes_below(sel[r])] = make_uint2(key[r], sub[r]);
    n += popc(sel[r]);
  }
  __builtin_amdgcn_wave_barrier();
  const uint2 v = lane < n ? s.stage[lane] : make_uint2(0u, 0u);
  __builtin_amdgcn_wave_barrier();
  out_key = v.x;
  out_id = v.y;
  return n;
}

// Merges the buffered candidate groups into the running top-K (lanes 0..K-1).
template <typename T, int RB>
__device__ __forceinline__ void flush_buffer(WaveLds& s, int nbuf, int64_t c0, int64_t c1, uint32_t tau, int K,
                                             int lane, uint32_t& cur_key, uint32_t& cur_id) {
  constexpr int EPG = Traits<T>::kPer;
  uint32_t key[RB + 1], sub[RB + 1];
  uint64_t live[RB + 1], sel[RB + 1];
  key[0] = cur_key;
  sub[0] = cur_id;
  live[0] = ballot(cur_key != 0);
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int e = r * kWave + lane;
    const int g = e / EPG, j = e % EPG;
    uint32_t k = 0, id = 0;
    if (g < nbuf) {
      const uint32_t word = reinterpret_cast<const uint32_t*>(&s.data[g])[j * 4 / EPG];
      const uint32_t bits = EPG == 8 ? (word >> (16 * (j & 1))) & 0xFFFFu : word;
      const int64_t gid = c0 + s.base[g] + j;
      if (gid < c1) {
        k = Traits<T>::key_bits(bits);
        id = static_cast<uint32_t>(gid);
        if (k < tau) k = 0;  // below the chunk's K-th largest: never selected
      }
    }
    key[r + 1] = k;
    sub[r + 1] = id;
    live[r + 1] = ballot(k != 0);
  }
  wave_select<RB + 1>(key, sub, live, K, Traits<T>::kKeyBits, sel);
  compact<RB + 1>(s, key, sub, sel, lane, cur_key, cur_id);
}

template <typename T>
__device__ __forceinline__ void flush(WaveLds& s, int nbuf, int64_t c0, int64_t c1, uint32_t tau, int K, int lane,
                                      uint32_t& cur_key, uint32_t& cur_id) {
  constexpr int EPG = Traits<T>::kPer;
  if (nbuf == 0) return;
  const int elems = nbuf * EPG;
  if (elems <= kWave)
    flush_buffer<T, 1>(s, nbuf, c0, c1, tau, K, lane, cur_key, cur_id);
  else if (elems <= 2 * kWave)
    flush_buffer<T, 2>(s, nbuf, c0, c1, tau, K, lane, cur_key, cur_id);
  else if (elems <= 4 * kWave)
    flush_buffer<T, 4>(s, nbuf, c0, c1, tau, K, lane, cur_key, cur_id);
  else
    flush_buffer<T, kCapGroups * EPG / kWave>(s, nbuf, c0, c1, tau, K, lane, cur_key, cur_id);
}

// The last wave of a row: merges the P partial results into LSE and the sorted top-K.
template <typename T>
__device__ void merge_row(int64_t row, int P, int K, int lane, WaveLds& s, const uint64_t* __restrict__ part_ms,
                          const uint64_t* __restrict__ part_ent, int32_t* __restrict__ cand_ids,
                          float* __restrict__ cand_logit, float* __restrict__ cand_logprob, float* __restrict__ lse) {
  const uint64_t* ms = part_ms + row * P;
  float m = neg_inf();
  for (int p = lane; p < P; p += kWave) m = fmaxf(m, __uint_as_float(static_cast<uint32_t>(load_agent(&ms[p]))));
  m = wave_max(m);
  float sum = 0.f;
  for (int p = lane; p < P; p += kWave) {
    const uint64_t v = load_agent(&ms[p]);
    const float pm = __uint_as_float(static_cast<uint32_t>(v));
    const float ps = __uint_as_float(static_cast<uint32_t>(v >> 32));
    if (pm != neg_inf()) sum += ps * fast_exp2((pm - m) * kLog2e);
  }
  sum = wave_sum(sum);
  const float l = (m == neg_inf()) ? neg_inf() : m + fast_log2(sum) * kLn2;

  constexpr int RB = 4;
  const uint64_t* ent = part_ent + row * static_cast<int64_t>(P) * K;
  const int total = P * K;
  uint32_t cur_key = 0, cur_id = 0;
  for (int base = 0; base < total; base += RB * kWave) {
    uint32_t key[RB + 1], sub[RB + 1];
    uint64_t live[RB + 1], sel[RB + 1];
    key[0] = cur_key;
    sub[0] = cur_id;
    live[0] = ballot(cur_key != 0);
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int e = base + r * kWave + lane;
      uint32_t k = 0, id = 0;
      if (e < total) {
        const uint64_t v = load_agent(&ent[e]);
        k = static_cast<uint32_t>(v);
        id = static_cast<uint32_t>(v >> 32);
      }
      key[r + 1] = k;
      sub[r + 1] = id;
      live[r + 1] = ballot(k != 0);
    }
    wave_select<RB + 1>(key, sub, live, K, Traits<T>::kKeyBits, sel);
    compact<RB + 1>(s, key, sub, sel, lane, cur_key, cur_id);
  }
  // Position of each selected entry in the (value desc, id asc) order.
  int rank = 0;
  for (int j = 0; j < K; ++j) {
    const uint32_t kj = __builtin_amdgcn_readlane(cur_key, j);
    const uint32_t ij = __builtin_amdgcn_readlane(cur_id, j);
    rank += (kj > cur_key) || (kj == cur_key && ij < cur_id);
  }
  if (lane < K) {
    const int64_t o = row * K + rank;
    const float v = Traits<T>::from_key(cur_key);
    cand_ids[o] = static_cast<int32_t>(cur_id);
    cand_logit[o] = v;
    if (cand_logprob) cand_logprob[o] = v - l;
  }
  if (lane == 0 && lse) lse[row] = l;
}

template <typename T, bool kAligned>
__global__ __launch_bounds__(kWave* kWavesPerBlock) void topk_sweep_kernel(
    const T* __restrict__ logits, int gamma, int64_t V, int64_t stride_b, int64_t stride_i, int K, int P,
    int64_t Q, uint32_t* __restrict__ counters, uint64_t* __restrict__ part_ms, uint64_t* __restrict__ part_ent,
    int32_t* __restrict__ cand_ids, float* __restrict__ cand_logit, float* __restrict__ cand_logprob,
    float* __restrict__ lse) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int64_t CH = static_cast<int64_t>(kGroups) * kWave * EPG;
  __shared__ WaveLds lds[kWavesPerBlock];

  const int w = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w;
  if (q >= Q) return;
  WaveLds& s = lds[w];
  const int64_t row = q / P;
  const int chunk = static_cast<int>(q - row * P);
  const int64_t b = row / gamma, i = row - b * gamma;
  const T* rp = logits + b * stride_b + i * stride_i;
  const int64_t c0 = chunk * CH;
  const int64_t c1 = c0 + CH < V ? c0 + CH : V;

  // 1. Stream the chunk into registers: group g of this lane covers elements
  //    c0 + (g*64 + lane)*EPG .. +EPG, so every load instruction reads 1 KB contiguous.
  u32x4 data[kGroups];
  if (kAligned && c0 + CH <= V) {
#pragma unroll
    for (int g = 0; g < kGroups; ++g)
      data[g] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(rp + c0 + (g * kWave + lane) * EPG));
  } else {
#pragma unroll
    for (int g = 0; g < kGroups; ++g)
      data[g] = load_group_checked<T, kAligned>(rp, c0 + (g * kWave + lane) * EPG, c1);
  }

  // 2. Per group: maximum and exp-sum relative to it; fold into the lane's (max, sum).
  float gmax[kGroups];
  float lm = neg_inf(), ls = 0.f;
#pragma unroll
  for (int g = 0; g < kGroups; ++g) {
    float x[EPG];
#pragma unroll
    for (int j = 0; j < EPG; ++j) x[j] = Traits<T>::elem(data[g], j);
    float gm = x[0];
#pragma unroll
    for (int j = 1; j < EPG; ++j) gm = fmaxf(gm, x[j]);
    gmax[g] = gm;
    if (gm != neg_inf()) {
      const float off = gm * kLog2e;
      float gs = 0.f;
#pragma unroll
      for (int j = 0; j < EPG; ++j) gs += fast_exp2(fmaf(x[j], kLog2e, -off));
      if (gm > lm) {
        ls = fmaf(ls, fast_exp2((lm - gm) * kLog2e), gs);
        lm = gm;
      } else {
        ls = fmaf(gs, fast_exp2((gm - lm) * kLog2e), ls);
      }
    }
  }

  // 3. The chunk's (max, sum).
  const float wm = wave_max(lm);
  const float wsum = wave_sum((lm == neg_inf()) ? 0.f : ls * fast_exp2((lm - wm) * kLog2e));

  // 4. tau = K-th largest lane maximum (key 0 for lanes without elements).
  const bool lane_valid = c0 + static_cast<int64_t>(lane) * EPG < c1;
  const uint32_t lkey[1] = {lane_valid ? Traits<T>::key_value(lm) : 0u};
  const uint64_t all[1] = {~0ull};
  const uint32_t tau = wave_kth_largest<1>(lkey, all, K, Traits<T>::kKeyBits);

  // 5. Groups whose maximum reaches tau can hold a top-K element.  They go to the LDS
  //    buffer in rounds of at most kCapGroups groups; each round is merged into the
  //    running top-K held in lanes 0..K-1.  Typical chunks need one round.
  uint32_t pending = 0;
#pragma unroll
  for (int g = 0; g < kGroups; ++g) {
    const int64_t rel = static_cast<int64_t>(g * kWave + lane) * EPG;
    if (c0 + rel < c1 && Traits<T>::key_value(gmax[g]) >= tau) pending |= 1u << g;
  }
  uint32_t cur_key = 0, cur_id = 0;
  while (ballot(pending != 0)) {
    int nbuf = 0;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
      const bool hit = (pending >> g) & 1u;
      const uint64_t m = ballot(hit);
      if (m) {
        const int pos = nbuf + static_cast<int>(lanes_below(m));
        if (hit && pos < kCapGroups) {
          s.data[pos] = data[g];
          s.base[pos] = static_cast<uint32_t>((g * kWave + lane) * EPG);
          pending &= ~(1u << g);
        }
        nbuf = nbuf + popc(m) < kCapGroups ? nbuf + popc(m) : kCapGroups;
      }
    }
    __builtin_amdgcn_wave_barrier();
    flush<T>(s, nbuf, c0, c1, tau, K, lane, cur_key, cur_id);
  }

  // 6. Publish the partial result with stores that are coherent at device scope, and
  //    wait until they have completed before counting this chunk as done.
  if (lane < K) store_agent(&part_ent[q * K + lane], pack(cur_key, cur_id));
  if (lane == 0) store_agent(&part_ms[q], pack(__float_as_uint(wm), __float_as_uint(wsum)));
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);

  // 7. The last wave of the row to arrive merges the row; its loads are device-coherent
  //    too, so no cache-wide writeback or invalidation is needed.
  uint32_t prev = 0;
  if (lane == 0) prev = __hip_atomic_fetch_add(&counters[row], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  prev = __builtin_amdgcn_readfirstlane(prev);
  if (prev != static_cast<uint32_t>(P - 1)) return;
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  merge_row<T>(row, P, K, lane, s, part_ms, part_ent, cand_ids, cand_logit, cand_logprob, lse);
  if (lane == 0) __hip_atomic_store(&counters[row], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

}  // namespace

TopkPlan topk_plan(int B, int gamma, int64_t V, int K, int dtype) {
  TopkPlan p{};
  const int epg = dtype == 1 ? 8 : 4;
  p.chunk = kGroups * kWave * epg;
  p.parts = static_cast<int>((V + p.chunk - 1) / p.chunk);
  const size_t rows = static_cast<size_t>(B) * gamma;
  p.off_ms = align256(rows * sizeof(uint32_t));
  p.off_ent = p.off_ms + align256(rows * p.parts * sizeof(uint64_t));
  p.bytes = p.off_ent + align256(rows * p.parts * static_cast<size_t>(K) * sizeof(uint64_t));
  return p;
}

hipError_t launch_topk(const void* logits, int dtype, bool aligned, int B, int gamma, int64_t V, int64_t stride_b,
                       int64_t stride_i, int K, const TopkPlan& plan, void* workspace, int32_t* cand_ids,
                       float* cand_logit, float* cand_logprob, float* lse, hipStream_t stream) {
  const int64_t Q = static_cast<int64_t>(B) * gamma * plan.parts;
  const dim3 grid(static_cast<unsigned>((Q + kWavesPerBlock - 1) / kWavesPerBlock));
  const dim3 block(kWave * kWavesPerBlock);
  char* ws = static_cast<char*>(workspace);
  uint32_t* counters = reinterpret_cast<uint32_t*>(ws);
  uint64_t* ms = reinterpret_cast<uint64_t*>(ws + plan.off_ms);
  uint64_t* ent = reinterpret_cast<uint64_t*>(ws + plan.off_ent);
  if (dtype == 1) {
    const uint16_t* x = static_cast<const uint16_t*>(logits);
    if (aligned)
      hipLaunchKernelGGL((topk_sweep_kernel<uint16_t, true>), grid, block, 0, stream, x, gamma, V, stride_b, stride_i,
                         K, plan.parts, Q, counters, ms, ent, cand_ids, cand_logit, cand_logprob, lse);
    else
      hipLaunchKernelGGL((topk_sweep_kernel<uint16_t, false>), grid, block, 0, stream, x, gamma, V, stride_b,
                         stride_i, K, plan.parts, Q, counters, ms, ent, cand_ids, cand_logit, cand_logprob, lse);
  } else {
    const float* x = static_cast<const float*>(logits);
    if (aligned)
      hipLaunchKernelGGL((topk_sweep_kernel<float, true>), grid, block, 0, stream, x, gamma, V, stride_b, stride_i, K,
                         plan.parts, Q, counters, ms, ent, cand_ids, cand_logit, cand_logprob, lse);
    else
      hipLaunchKernelGGL((topk_sweep_kernel<float, false>), grid, block, 0, stream, x, gamma, V, stride_b, stride_i,
                         K, plan.parts, Q, counters, ms, ent, cand_ids, cand_logit, cand_logprob, lse);
  }
  return hipGetLastError();
}

}  // namespace ubt
