// Softmax statistics and top-K candidates of one logit row, run by one workgroup of 8
// waves: the device code shared by the top-K kernel and the one-launch draft step.
//
// Method / Unigram Proposer, Eq. (ubtree-unigram), q_i = softmax(u_i), and "Candidate
// Sets": C_i = the K tokens of largest q_i, ranked here on the logits (softmax is
// increasing) with ties to the lower token id.
//
// One HBM pass, one workgroup of 8 waves per row.  The row is cut into tiles of 64 lanes
// x 4 groups x 16 B (2048 bf16 or 1024 fp32 elements), dealt round-robin to the waves;
// each wave streams its tiles with the next one in flight (nontemporal 16-byte buffer
// loads addressed by a fixed lane offset plus a wave-uniform scalar base).  A ragged last
// tile rides in the same pipeline: loads past the row read zeros, which are masked to
// -inf.  A lane keeps a running (max, sum of exp(x - max)) whose max may trail the true
// one by a bounded slack, so most tiles need no rescale: one exp per element.  Waves
// with more tiles left get a higher issue priority, so the two workgroups that share a
// CU finish together instead of one starving the other.
//
// Top-K: a group can hold a top-K element only if its maximum reaches a threshold that
// is known to be at most the row's K-th largest element.  After every wave has reduced
// its first tile, the workgroup takes T = the K-th largest of the 64 column maxima of
// the lane maxima (K distinct groups reach it), found by counting; from then on only
// groups whose maximum reaches T are buffered in LDS.  At the end each wave stages its
// live elements (key >= T), ranks them by counting and publishes its top K, sorted, with
// its K-th key; wave 0 keeps the published candidates at or above the best K-th key
// (a lower bound of the row's K-th), ranks them by counting and writes the row's LSE and
// sorted top-K.  Radix selection is the fallback for more than 64 candidates, and a wave
// whose buffer overflows re-scans its tiles exactly.
#pragma once

#include "ubt_device.h"

namespace ubt {
namespace {

constexpr int kSubGroups = 4;     // 16-byte groups per lane per tile
constexpr int kWaves = 8;         // waves per workgroup
constexpr int kCapGroups = 64;    // LDS candidate-group buffer per wave

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
  __device__ static uint32_t key_bits(uint32_t bits) { return f32_key(__uint_as_float(bits)); }
  __device__ static uint32_t key_value(float f) { return f32_key(f); }
  __device__ static float from_key(uint32_t k) { return f32_key_value(k); }
  __device__ static void set_neg_inf(u32x4& v) { v = u32x4{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u}; }
  __device__ static void set_elem(u32x4& v, int j, uint32_t bits) { v[j] = bits; }
  __device__ static uint32_t load_elem(const float* p) { return __float_as_uint(*p); }
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

template <int CAP>
struct WaveLdsT {
  static constexpr int kCap = CAP;
  u32x4 data[CAP];     // buffered candidate groups
  uint32_t base[CAP];  // row index of each group's first element
  uint2 stage[kWave];         // compaction staging (key, id)
  uint64_t cand[kWave];       // live candidates as 64-bit order values
};
using WaveLds = WaveLdsT<kCapGroups>;

// Shared memory of one row's workgroup of up to MW waves.
template <int MW>
struct RowLdsT {
  WaveLds wave[MW];
  uint64_t part64[MW * kWave];  // wave w's top candidates, sorted, at [w*K, w*K + npart[w])
  int npart[MW];
  uint32_t thr2;                     // max over the waves of their K-th candidate key
  uint2 part[MW * kWave];        // (key, id) copy of part64 for the radix fallback
  float2 ms[MW];                 // each wave's (max, sum)
  uint32_t lane_max[MW * kWave]; // lane maxima (keys) of every wave's first tile
};
using RowLds = RowLdsT<kWaves>;

// A buffer resource covering one row: loads address it with a 32-bit offset in a scalar
// descriptor instead of a 64-bit address per lane, and offsets past the row read zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_resource(const void* row, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(row), 0, static_cast<int>(bytes), 0x00020000);
}

constexpr int kNontemporal = 2;  // cache policy of the streaming loads (read once)

// Loads the tile [c0, c0 + SUB) of an aligned row; bytes past the row read as zero.
// The lane's byte offset goes in the vector offset (the same register for every load of
// the pass) and the wave-uniform tile base in the scalar offset, so issuing a load writes
// no vector register other than its destination.
template <typename T>
__device__ __forceinline__ void load_full(u32x4 (&buf)[kSubGroups], __amdgpu_buffer_rsrc_t rsrc, int64_t c0,
                                          uint32_t lane_off) {
  constexpr int EPG = Traits<T>::kPer;
  const uint32_t base = static_cast<uint32_t>(c0 * sizeof(T));
  // Issued in group order (no reordering across the barriers): the wait for group g then
  // counts exactly the loads issued after it.
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g) {
    buf[g] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           rsrc, lane_off, base + g * kWave * EPG * sizeof(T), kNontemporal));
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Loads tile elements [c0, c0 + SUB) of a row that may end inside it or be
// unaligned; elements >= V read as -inf.  A 16-byte load that would cross the end of the
// row is replaced by element loads.
template <typename T, bool kAligned>
__device__ __forceinline__ void load_checked(u32x4 (&buf)[kSubGroups], __amdgpu_buffer_rsrc_t rsrc, const T* rp,
                                             int64_t c0, int64_t V, int lane) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * EPG;
  const int lim = static_cast<int>(V - c0 < SUB ? V - c0 : SUB);
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g) {
    const int r0 = (g * kWave + lane) * EPG;
    if (kAligned && r0 + EPG <= lim) {
      buf[g] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                             rsrc, static_cast<uint32_t>((c0 + r0) * sizeof(T)), 0, kNontemporal));
    } else {
      Traits<T>::set_neg_inf(buf[g]);
      for (int j = 0; j < EPG; ++j)
        if (r0 + j < lim) Traits<T>::set_elem(buf[g], j, Traits<T>::load_elem(rp + c0 + r0 + j));
    }
  }
}

// Sets the groups of a tile that lie at or past V to -inf (groups never straddle V when
// V * sizeof(T) is a multiple of 16, the only case that loads a ragged tile whole).
template <typename T>
__device__ __forceinline__ void mask_tail(u32x4 (&buf)[kSubGroups], int64_t c0, int64_t V, int lane) {
  constexpr int EPG = Traits<T>::kPer;
  const int64_t lane_e = c0 + lane * EPG;
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g)
    if (lane_e >= V - g * kWave * EPG) Traits<T>::set_neg_inf(buf[g]);
}

// Wave priority from the number of tiles this wave still has to stream: waves that are
// behind win the issue arbitration, so the waves sharing a CU finish together.
__device__ __forceinline__ void set_prio(int rem) {
  if (rem >= 6) __builtin_amdgcn_s_setprio(3);
  else if (rem >= 4) __builtin_amdgcn_s_setprio(2);
  else if (rem >= 2) __builtin_amdgcn_s_setprio(1);
  else __builtin_amdgcn_s_setprio(0);
}

// Compacts the selected entries (at most 64) into lanes 0.. of (out_key, out_id).
template <int R, class WL>
__device__ __forceinline__ void compact(WL& s, const uint32_t (&key)[R], const uint32_t (&sub)[R],
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
}

// Merges the buffered candidate groups into the running top-K (lanes 0..K-1), or, with
// kCarry false, selects the top K of the groups alone (the running top-K is empty).
// Elements whose key does not pass the threshold (key >= thr, or key > thr when strict)
// are dropped: they cannot be in the top K.
template <typename T, int RB, bool kCarry, class WL>
__device__ __forceinline__ void flush_buffer(WL& s, int g0, int nbuf, int64_t V, uint32_t thr, bool strict, int K,
                                             int lane, uint32_t& cur_key, uint32_t& cur_id) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int C = kCarry ? 1 : 0;
  uint32_t key[RB + C], sub[RB + C];
  uint64_t live[RB + C], sel[RB + C];
  if (kCarry) {
    key[0] = cur_key;
    sub[0] = cur_id;
    live[0] = ballot(cur_key != 0);
  }
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int e = r * kWave + lane;
    const int g = g0 + e / EPG, j = e % EPG;
    uint32_t k = 0, id = 0;
    if (g < nbuf) {
      const uint32_t word = reinterpret_cast<const uint32_t*>(&s.data[g])[j * 4 / EPG];
      const uint32_t bits = EPG == 8 ? (word >> (16 * (j & 1))) & 0xFFFFu : word;
      const int64_t gid = static_cast<int64_t>(s.base[g]) + j;
      if (gid < V) {
        k = Traits<T>::key_bits(bits);
        id = static_cast<uint32_t>(gid);
        if (strict ? k <= thr : k < thr) k = 0;
      }
    }
    key[r + C] = k;
    sub[r + C] = id;
    live[r + C] = ballot(k != 0);
  }
  wave_select<RB + C>(key, sub, live, K, Traits<T>::kKeyBits, sel);
  compact<RB + C>(s, key, sub, sel, lane, cur_key, cur_id);
}

// Merges nbuf buffered groups into the running top-K; returns the new (key, id) pair of
// this lane (lanes 0..K-1 hold the top K).  kFresh: the running top-K is empty.
template <typename T, bool kFresh, class WL>
__device__ __forceinline__ uint2 flush(WL& s, int nbuf, int64_t V, uint32_t thr, bool strict, int K, int lane,
                                       uint32_t cur_key, uint32_t cur_id) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int kSlice = 4 * kWave / EPG;  // groups per selection pass (four register rows)
  for (int g0 = 0; g0 < nbuf; g0 += kSlice) {
    const int elems = (nbuf - g0 < kSlice ? nbuf - g0 : kSlice) * EPG;
    if (kFresh && g0 == 0) {
      if (elems <= kWave)
        flush_buffer<T, 1, false>(s, g0, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
      else if (elems <= 2 * kWave)
        flush_buffer<T, 2, false>(s, g0, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
      else
        flush_buffer<T, 4, false>(s, g0, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
    } else {
      if (elems <= kWave)
        flush_buffer<T, 1, true>(s, g0, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
      else if (elems <= 2 * kWave)
        flush_buffer<T, 2, true>(s, g0, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
      else
        flush_buffer<T, 4, true>(s, g0, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
    }
  }
  return make_uint2(cur_key, cur_id);
}

// The top K of the waves' candidates part[0..total), total <= 64 R, into lanes 0..K-1.
template <typename T, int R, class WL>
__device__ __forceinline__ void merge_parts(const uint2* part, int total, int K, int lane, WL& s,
                                            uint32_t& cur_key, uint32_t& cur_id) {
  uint32_t key[R], sub[R];
  uint64_t live[R], sel[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int e = r * kWave + lane;
    const uint2 v = e < total ? part[e] : make_uint2(0u, 0u);
    key[r] = v.x;
    sub[r] = v.y;
    live[r] = ballot(v.x != 0);
  }
  wave_select<R>(key, sub, live, K, Traits<T>::kKeyBits, sel);
  compact<R>(s, key, sub, sel, lane, cur_key, cur_id);
}


// 64-bit order value of a candidate: larger is better (key desc, then id asc).
__device__ __forceinline__ uint64_t cand_order(uint32_t key, uint32_t id) {
  return (static_cast<uint64_t>(key) << 32) | static_cast<uint32_t>(~id);
}
// Number of the n order values at v[0..n) (LDS, 16-byte aligned, 64 entries readable)
// greater than `mine`.  Eight entries per round trip.
// Four independent counts, so that the compares of one round trip do not wait on each
// other (a lone wave would otherwise stall on every add).
__device__ __forceinline__ int count_above(const uint64_t* v, int n, uint64_t mine) {
  int c[4] = {0, 0, 0, 0};
  for (int j0 = 0; j0 < n; j0 += 8) {
    ulonglong2 p[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) p[q] = *reinterpret_cast<const ulonglong2*>(v + j0 + 2 * q);
#pragma unroll
    for (int q = 0; q < 4; ++q) c[q] += (j0 + 2 * q < n && p[q].x > mine) + (j0 + 2 * q + 1 < n && p[q].y > mine);
  }
  return (c[0] + c[1]) + (c[2] + c[3]);
}
// Stages the buffered elements with key >= thr to s.cand (in buffer order); returns how
// many there are (only the first 64 are staged).
template <typename T, class WL>
__device__ __forceinline__ int stage_live(WL& s, int nbuf, int64_t V, uint32_t thr, int lane) {
  constexpr int EPG = Traits<T>::kPer;
  const int total = nbuf * EPG;
  int n = 0;
  for (int e0 = 0; e0 < total; e0 += kWave) {
    const int e = e0 + lane;
    uint32_t k = 0, id = 0;
    if (e < total) {
      const int g = e / EPG, j = e % EPG;
      const uint32_t word = reinterpret_cast<const uint32_t*>(&s.data[g])[j * 4 / EPG];
      const uint32_t bits = EPG == 8 ? (word >> (16 * (j & 1))) & 0xFFFFu : word;
      const int64_t gid = static_cast<int64_t>(s.base[g]) + j;
      if (gid < V) {
        k = Traits<T>::key_bits(bits);
        id = static_cast<uint32_t>(gid);
        if (k < thr) k = 0;
      }
    }
    const uint64_t m = ballot(k != 0);
    const int pos = n + static_cast<int>(lanes_below(m));
    if (k != 0 && pos < kWave) s.cand[pos] = cand_order(k, id);
    n += popc(m);
  }
  return n;
}

// Smallest key among the K candidates held in lanes 0..K-1.
__device__ __forceinline__ uint32_t kth_key(uint32_t cur_key, int K, int lane) {
  uint32_t mn = lane < K ? cur_key : 0xFFFFFFFFu;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) mn = min(mn, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mn), o, kWave)));
  return mn;
}

// Per-wave running state of the streaming pass.
struct WaveState {
  float lm, ls;   // lane's running max and exp-sum relative to it
  uint32_t thr;   // candidate threshold key (0 = none): groups need max key >= thr
  int nbuf;       // groups waiting in the LDS buffer
  bool overflow;  // a group that passed could not be buffered
  // K > 16: a full buffer is merged into a running top K instead (lanes 0..K-1 of
  // cur_key/cur_id), and the threshold tightens to its K-th key (strictly, once K are held:
  // later elements carry larger ids).
  bool strict, merged;
  uint32_t cur_key, cur_id;
};

// Buffers the groups of pending that pass.  kBig (K > 16): a full buffer is merged into
// the running top K, the threshold tightened, and the rest re-filtered, until every
// passing group is held.  Otherwise a group that does not fit sets `overflow` (exact
// re-scan at the end).
template <typename T, bool kBig, class WL>
__device__ __forceinline__ void push_groups(const u32x4 (&buf)[kSubGroups], const float (&gmax)[kSubGroups],
                                            uint32_t pending, int64_t c0, int64_t V, int K, int lane, WL& s,
                                            WaveState& st);

// Max and exp-sum of one tile, folded into the lane's running (lm, ls): ls is the
// sum of exp(x - lm) over the lane's elements so far, where lm may trail the lane's true
// maximum by up to kSlack (terms stay below e^kSlack, far from fp32 overflow).  lm is
// raised, with one rescale of ls, only when a tile would break that bound.
constexpr float kSlack = 32.f;
template <typename T>
__device__ __forceinline__ float reduce_sub(const u32x4 (&buf)[kSubGroups], float (&gmax)[kSubGroups], float& lm,
                                            float& ls) {
  constexpr int EPG = Traits<T>::kPer;
  float x[kSubGroups][EPG];
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g)
#pragma unroll
    for (int j = 0; j < EPG; ++j) x[g][j] = Traits<T>::elem(buf[g], j);
  // maximum() needs no NaN canonicalisation of its inputs (maxnum does); logits are
  // never NaN, so the two agree here.
  float sub_max;
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g) {
    float gm = x[g][0];
#pragma unroll
    for (int j = 1; j + 1 < EPG; j += 2)
      gm = __builtin_elementwise_maximum(gm, __builtin_elementwise_maximum(x[g][j], x[g][j + 1]));
    if (EPG % 2 == 0) gm = __builtin_elementwise_maximum(gm, x[g][EPG - 1]);
    gmax[g] = gm;
    sub_max = g == 0 ? gm : __builtin_elementwise_maximum(sub_max, gm);
  }
  const float nlm = fmaxf(lm, sub_max - kSlack);
  const float f = fast_exp2((lm - nlm) * kLog2e);
  ls = lm == nlm ? ls : ls * f;  // lm == nlm == -inf keeps ls (= 0)
  lm = nlm;
  const float off = nlm == neg_inf() ? 0.f : nlm * kLog2e;  // every x is -inf while nlm is
  float s0 = fast_exp2(fmaf(x[0][0], kLog2e, -off)), s1 = fast_exp2(fmaf(x[0][1], kLog2e, -off));
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g)
#pragma unroll
    for (int j = (g == 0 ? 2 : 0); j < EPG; j += 2) {
      s0 += fast_exp2(fmaf(x[g][j], kLog2e, -off));
      s1 += fast_exp2(fmaf(x[g][j + 1], kLog2e, -off));
    }
  ls += s0 + s1;
  return sub_max;
}

// Group maxima of one tile (re-scan path).
template <typename T>
__device__ __forceinline__ void group_max_sub(const u32x4 (&buf)[kSubGroups], float (&gmax)[kSubGroups]) {
  constexpr int EPG = Traits<T>::kPer;
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g) {
    float gm = Traits<T>::elem(buf[g], 0);
#pragma unroll
    for (int j = 1; j < EPG; ++j) gm = fmaxf(gm, Traits<T>::elem(buf[g], j));
    gmax[g] = gm;
  }
}

// True if any lane of the wave has a group of a full tile whose maximum reaches thr.
template <typename T>
__device__ __forceinline__ bool any_pass_full(const float (&gmax)[kSubGroups], uint32_t thr) {
  const float thr_v = thr == 0 ? neg_inf() : Traits<T>::from_key(thr);
  uint64_t m = 0;
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g) m |= ballot(gmax[g] >= thr_v);
  return m != 0;
}

// Bit g set if group g of this lane is inside the row and its maximum passes the
// threshold (key >= thr, or key > thr when strict; thr = 0 passes everything).
template <typename T>
__device__ __forceinline__ uint32_t passing_groups(const float (&gmax)[kSubGroups], int64_t c0, int64_t V,
                                                   uint32_t thr, bool strict, int lane) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * EPG;
  const float thr_v = Traits<T>::from_key(thr);
  const bool full = c0 + SUB <= V;
  const int lim = full ? static_cast<int>(SUB) : static_cast<int>(V - c0);
  // One register for the lane's offset; the group's part of it is folded into the limit.
  const int lane_e = lane * EPG;
  uint32_t pending = 0;
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g) {
    const bool valid = full || lane_e < lim - g * kWave * EPG;
    const bool pass = thr == 0 || (strict ? gmax[g] > thr_v : gmax[g] >= thr_v);
    if (valid && pass) pending |= 1u << g;
  }
  return pending;
}

// Appends this lane's pending groups to the wave's LDS buffer; returns the groups that
// did not fit.
template <typename T, class WL>
__device__ __forceinline__ uint32_t buffer_groups(const u32x4 (&buf)[kSubGroups], uint32_t pending, int64_t c0,
                                                  int lane, WL& s, int& nbuf) {
  constexpr int EPG = Traits<T>::kPer;
#pragma unroll
  for (int g = 0; g < kSubGroups; ++g) {
    const bool hit = (pending >> g) & 1u;
    const uint64_t m = ballot(hit);
    if (m) {
      const int pos = nbuf + static_cast<int>(lanes_below(m));
      if (hit && pos < WL::kCap) {
        s.data[pos] = buf[g];
        s.base[pos] = static_cast<uint32_t>(c0) + static_cast<uint32_t>((g * kWave + lane) * EPG);
        pending &= ~(1u << g);
      }
      nbuf = nbuf + popc(m) < WL::kCap ? nbuf + popc(m) : WL::kCap;
    }
  }
  return pending;
}

// Exact fallback for a wave whose buffer overflowed (e.g. rows with long runs of equal
// values): re-reads its tiles and keeps a running top-K, merging the buffer each
// time it fills and tightening the threshold once K candidates are held (later groups
// carry larger ids, so they must beat the K-th candidate strictly).
template <typename T, bool kAligned, class WL>
__device__ uint2 rescan(__amdgpu_buffer_rsrc_t rsrc, const T* rp, int64_t first, int64_t nsub, int nw, int64_t V,
                        uint32_t thr, int K, int lane, WL& s) {
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * Traits<T>::kPer;
  uint32_t cur_key = 0, cur_id = 0;
  bool strict = false;
  int nbuf = 0;
  for (int64_t sc = first; sc < nsub; sc += nw) {
    u32x4 buf[kSubGroups];
    float gmax[kSubGroups];
    load_checked<T, kAligned>(buf, rsrc, rp, sc * SUB, V, lane);
    group_max_sub<T>(buf, gmax);
    uint32_t pending = passing_groups<T>(gmax, sc * SUB, V, thr, strict, lane);
    while (ballot(pending != 0)) {
      pending = buffer_groups<T>(buf, pending, sc * SUB, lane, s, nbuf);
      if (ballot(pending != 0)) {
        __builtin_amdgcn_wave_barrier();
        const uint2 c = flush<T, false>(s, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
        cur_key = c.x;
        cur_id = c.y;
        nbuf = 0;
      }
    }
    if (nbuf > 0) {
      __builtin_amdgcn_wave_barrier();
      const uint2 c = flush<T, false>(s, nbuf, V, thr, strict, K, lane, cur_key, cur_id);
      cur_key = c.x;
      cur_id = c.y;
      nbuf = 0;
    }
    if (popc(ballot(cur_key != 0)) >= K) {
      const uint32_t mn = kth_key(cur_key, K, lane);
      if (mn > thr || (mn == thr && !strict)) {
        thr = mn;
        strict = true;
      }
    }
  }
  return make_uint2(cur_key, cur_id);
}

template <typename T, bool kBig, class WL>
__device__ __forceinline__ void push_groups(const u32x4 (&buf)[kSubGroups], const float (&gmax)[kSubGroups],
                                            uint32_t pending, int64_t c0, int64_t V, int K, int lane, WL& s,
                                            WaveState& st) {
  pending = buffer_groups<T>(buf, pending, c0, lane, s, st.nbuf);
  if (!ballot(pending != 0)) return;
  if (!kBig) {
    st.overflow = true;
    return;
  }
  do {
    __builtin_amdgcn_wave_barrier();
    const uint2 c = flush<T, false>(s, st.nbuf, V, st.thr, st.strict, K, lane, st.cur_key, st.cur_id);
    st.cur_key = c.x;
    st.cur_id = c.y;
    st.nbuf = 0;
    st.merged = true;
    __builtin_amdgcn_wave_barrier();
    if (popc(ballot(st.cur_key != 0)) >= K) {
      const uint32_t mn = kth_key(st.cur_key, K, lane);
      if (mn > st.thr || (mn == st.thr && !st.strict)) {
        st.thr = mn;
        st.strict = true;
      }
    }
    pending &= passing_groups<T>(gmax, c0, V, st.thr, st.strict, lane);
    pending = buffer_groups<T>(buf, pending, c0, lane, s, st.nbuf);
  } while (ballot(pending != 0));
}

// Where a row's results go.  With `coherent`, the stores are device-coherent (they reach
// the point of coherence of all XCDs), for a reader in another workgroup of the same
// launch that waits on a flag.
struct RowOut {
  int32_t* cand_ids;
  float* cand_logit;
  float* cand_logprob;
  float* lse;
  bool coherent;
  template <typename P>
  __device__ __forceinline__ void put(P* p, uint32_t bits) const {
    uint32_t* q = reinterpret_cast<uint32_t*>(p);
    if (coherent)
      __hip_atomic_store(q, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      *q = bits;
  }
};

// The streaming pass over the row at rp (V elements) by wave w of nw: the running
// (max, exp-sum) of each lane and the groups that reach the candidate threshold, in the
// wave's buffer s (with kBig, also a running top K).  lane_max (nw * 64 words of LDS)
// receives the lane maxima of the first tiles; the threshold is agreed on after one
// __syncthreads of the workgroup.
template <typename T, bool kAligned, int MW, bool kBig, class WL>
__device__ __forceinline__ void stream_row(WL& s, uint32_t* lane_max, const T* __restrict__ rp, int64_t V, int K,
                                           int nw, int w, int lane, __amdgpu_buffer_rsrc_t rsrc, WaveState& st) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * EPG;
  const int64_t nsub = (V + SUB - 1) / SUB;
  const uint32_t lane_off = static_cast<uint32_t>(lane * EPG * sizeof(T));
  st = WaveState{neg_inf(), 0.f, 0u, 0, false, false, false, 0u, 0u};
  u32x4 bufA[kSubGroups], bufB[kSubGroups];
  float gmax[kSubGroups];
  // Tiles [0, nfull) stream through the pipeline (aligned rows only, with the ragged last
  // tile when V * sizeof(T) is a multiple of 16); the others go through checked loads.
  const int64_t nfull0 = kAligned ? V / SUB : 0;
  const int64_t nfull = kAligned && (V * static_cast<int64_t>(sizeof(T))) % 16 == 0 ? nsub : nfull0;
  const int64_t last_c0 = (nfull > nfull0) ? (nsub - 1) * SUB : -1;
  int64_t sc = w;

  // First tile of every wave, then one workgroup-wide threshold.  Only the first tile is
  // requested up front: every wave of the launch needs it before its workgroup can agree
  // on a threshold, so those requests must not queue behind other waves' prefetches.
  // The second follows as soon as it has arrived.
  if (sc < nfull) {
    load_full<T>(bufA, rsrc, sc * SUB, lane_off);
    uint32_t x = bufA[kSubGroups - 1][0];
    asm volatile("" : "+v"(x));  // the first tile has arrived
    __builtin_amdgcn_sched_barrier(0);
  }
  if (sc + nw < nfull) load_full<T>(bufB, rsrc, (sc + nw) * SUB, lane_off);
  {
    uint32_t lkey = 0;
    if (sc * SUB == last_c0) mask_tail<T>(bufA, sc * SUB, V, lane);
    if (sc < nfull) lkey = Traits<T>::key_value(reduce_sub<T>(bufA, gmax, st.lm, st.ls));
    lane_max[w * kWave + lane] = lkey;
  }
  __syncthreads();
  if (kBig) {
    // T = (a lower bound of) the K-th largest of all the lane maxima: K of them, maxima of
    // disjoint elements, reach it.  For large K this is far tighter than the K-th column
    // maximum (each column maximum covers all the waves' lanes).
    uint32_t lk[MW];
    uint64_t lv[MW];
#pragma unroll
    for (int j = 0; j < MW; ++j) {
      lk[j] = j < nw ? lane_max[j * kWave + lane] : 0u;
      lv[j] = ballot(lk[j] != 0u);
    }
    st.thr = wave_threshold<MW>(lk, lv, K, K + K / 4);
  } else {
    // T = the K-th largest of the 64 column maxima (lane l's largest lane maximum over the
    // waves): K distinct groups reach it, so it is a lower bound of the row's K-th largest
    // element.  Each lane counts the column maxima above its own.
    uint32_t cm = 0;
    for (int j = 0; j < nw; ++j) cm = max(cm, lane_max[j * kWave + lane]);
    uint32_t* sv = reinterpret_cast<uint32_t*>(s.stage);
    sv[lane] = cm;
    __builtin_amdgcn_wave_barrier();
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < kWave; j += 4) {
      const uint4 v = *reinterpret_cast<const uint4*>(&sv[j]);
      cnt += (v.x > cm) + (v.y > cm) + (v.z > cm) + (v.w > cm);
    }
    __builtin_amdgcn_wave_barrier();
    const int n_live = popc(ballot(cm != 0));
    st.thr = n_live < K ? 0u : wave_umin(cm != 0 && cnt < K ? cm : ~0u);
  }
  if (sc < nfull) {
    const uint32_t p = passing_groups<T>(gmax, sc * SUB, V, st.thr, false, lane);
    if (ballot(p != 0)) push_groups<T, kBig>(bufA, gmax, p, sc * SUB, V, K, lane, s, st);
  }
  sc += nw;

  // Reduces tile c0 and buffers its groups that reach the threshold.
  auto consume = [&](u32x4 (&buf)[kSubGroups], int64_t c0) {
    if (c0 == last_c0) mask_tail<T>(buf, c0, V, lane);
    reduce_sub<T>(buf, gmax, st.lm, st.ls);
    if (!st.overflow && any_pass_full<T>(gmax, st.thr)) {
      const uint32_t p = passing_groups<T>(gmax, c0, V, st.thr, st.strict, lane);
      if (ballot(p != 0)) push_groups<T, kBig>(buf, gmax, p, c0, V, K, lane, s, st);
    }
  };
  // The remaining tiles, the next one always in flight; the last tile issues no load.
  if (sc < nfull) {
    int left = static_cast<int>((nfull - 1 - sc) / nw);  // tiles after the current one
    for (;;) {
      if (left == 0) {
        consume(bufB, sc * SUB);
        break;
      }
      set_prio(left--);
      load_full<T>(bufA, rsrc, (sc + nw) * SUB, lane_off);
      consume(bufB, sc * SUB);
      sc += nw;
      if (left == 0) {
        consume(bufA, sc * SUB);
        break;
      }
      set_prio(left--);
      load_full<T>(bufB, rsrc, (sc + nw) * SUB, lane_off);
      consume(bufA, sc * SUB);
      sc += nw;
    }
  }

  __builtin_amdgcn_s_setprio(3);
  // Ragged or unaligned tiles: this wave's share of [nfull, nsub).
  for (int64_t sr = nfull + ((w - nfull % nw) + nw) % nw; sr < nsub; sr += nw) {
    load_checked<T, kAligned>(bufA, rsrc, rp, sr * SUB, V, lane);
    reduce_sub<T>(bufA, gmax, st.lm, st.ls);
    if (!st.overflow) {
      const uint32_t p = passing_groups<T>(gmax, sr * SUB, V, st.thr, st.strict, lane);
      if (ballot(p != 0)) push_groups<T, kBig>(bufA, gmax, p, sr * SUB, V, K, lane, s, st);
    }
  }

}

// The row at rp (V elements) of global row index `row`; the workgroup has up to MW waves
// and `lds` is its shared memory.  Writes cand_*[row * K, row * K + K) and lse[row].
template <typename T, bool kAligned, int MW = kWaves, bool kBig = false>
__device__ __forceinline__ void sweep_row(RowLdsT<MW>& lds, const T* __restrict__ rp, int64_t V, int K, int64_t row,
                                          const RowOut& out) {
  constexpr int EPG = Traits<T>::kPer;
  constexpr int64_t SUB = static_cast<int64_t>(kSubGroups) * kWave * EPG;
  const int nw = blockDim.x / kWave;
  // Wave-uniform, and known to be: the tile indices and offsets derived from it
  // then live in scalar registers.
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const __amdgpu_buffer_rsrc_t rsrc = row_resource(rp, static_cast<uint32_t>(V * static_cast<int64_t>(sizeof(T))));
  const int64_t nsub = (V + SUB - 1) / SUB;
  WaveLds& s = lds.wave[w];
  if (threadIdx.x == 0) lds.thr2 = 0;  // published by the barrier inside the pass
  WaveState st;
  stream_row<T, kAligned, MW, kBig>(s, lds.lane_max, rp, V, K, nw, w, lane, rsrc, st);

  // This wave's live candidates (key >= the threshold) in s.cand: staged straight from
  // the buffer, or, when there are more than 64 of them or the buffer overflowed, the top
  // K picked by the radix selection.
  int n = 0;
  if (!st.overflow && !(kBig && st.merged)) n = st.nbuf > 0 ? stage_live<T>(s, st.nbuf, V, st.thr, lane) : 0;
  if (st.overflow || (kBig && st.merged) || n > kWave) {
    uint32_t ck = 0, ci = 0;
    if (kBig && st.merged) {
      // The running top K plus what the buffer still holds.
      __builtin_amdgcn_wave_barrier();
      const uint2 c = st.nbuf > 0 ? flush<T, false>(s, st.nbuf, V, st.thr, st.strict, K, lane, st.cur_key, st.cur_id)
                                  : make_uint2(st.cur_key, st.cur_id);
      ck = c.x;
      ci = c.y;
    } else if (!st.overflow) {
      __builtin_amdgcn_wave_barrier();
      const uint2 c = flush<T, true>(s, st.nbuf, V, st.thr, false, K, lane, 0u, 0u);
      ck = c.x;
      ci = c.y;
    } else {
      const uint2 c = rescan<T, kAligned>(rsrc, rp, w, nsub, nw, V, st.thr, K, lane, s);
      ck = c.x;
      ci = c.y;
    }
    const uint64_t m = ballot(ck != 0);
    __builtin_amdgcn_wave_barrier();
    if (ck != 0) s.cand[lanes_below(m)] = cand_order(ck, ci);
    n = popc(m);
  }
  __builtin_amdgcn_wave_barrier();
  {
    // Rank of each candidate among the wave's: the first K in rank order are the wave's
    // top K, written sorted; the K-th one's key bounds the row's K-th from below.
    const uint64_t mine = lane < n ? s.cand[lane] : 0ull;
    const int r = lane < n ? count_above(s.cand, n, mine) : kWave;
    if (r < K) lds.part64[w * K + r] = mine;
    if (n >= K && r == K - 1) atomicMax(&lds.thr2, static_cast<uint32_t>(mine >> 32));
    if (lane == 0) lds.npart[w] = n < K ? n : K;
  }

  const float wm = wave_max(st.lm);
  const float wsum = wave_sum((st.lm == neg_inf()) ? 0.f : st.ls * fast_exp2((st.lm - wm) * kLog2e));
  if (lane == 0) lds.ms[w] = make_float2(wm, wsum);
  __syncthreads();
  if (w != 0) return;

  float2 ms[MW];
#pragma unroll
  for (int j = 0; j < MW; ++j) ms[j] = lds.ms[j];
  float m = neg_inf();
#pragma unroll
  for (int j = 0; j < MW; ++j) m = j < nw ? fmaxf(m, ms[j].x) : m;
  float e = 0.f;
#pragma unroll
  for (int j = 0; j < MW; ++j)
    if (j < nw && ms[j].x != neg_inf()) e += ms[j].y * fast_exp2((ms[j].x - m) * kLog2e);
  const float l = (m == neg_inf()) ? neg_inf() : m + fast_log2(e) * kLn2;

  // The waves' candidates at or above the best K-th key (a lower bound of the row's K-th
  // largest), gathered into s.cand; more than 64 of them fall back to the radix merge.
  const uint32_t t3 = lds.thr2;
  const int slots = nw * K;
  int nf = 0;
  for (int e0 = 0; e0 < slots; e0 += kWave) {
    const int e = e0 + lane;
    uint64_t v = 0;
    if (e < slots) {
      const int ww = e / K, j = e - ww * K;
      if (j < lds.npart[ww]) v = lds.part64[e];
      if (static_cast<uint32_t>(v >> 32) < t3) v = 0;
    }
    const uint64_t msk = ballot(v != 0);
    const int pos = nf + static_cast<int>(lanes_below(msk));
    if (v != 0 && pos < kWave) s.cand[pos] = v;
    nf += popc(msk);
  }
  __builtin_amdgcn_wave_barrier();
  uint64_t mine = 0;
  int r = kWave;
  if (nf <= kWave) {
    mine = lane < nf ? s.cand[lane] : 0ull;
    r = lane < nf ? count_above(s.cand, nf, mine) : kWave;
  } else {
    // Rare (heavy ties): radix selection over all the waves' candidates.
    for (int e = lane; e < slots; e += kWave) {
      const int ww = e / K, j = e - ww * K;
      const uint64_t v = j < lds.npart[ww] ? lds.part64[e] : 0ull;
      lds.part[e] = make_uint2(static_cast<uint32_t>(v >> 32), ~static_cast<uint32_t>(v));
    }
    __builtin_amdgcn_wave_barrier();
    uint32_t ck = 0, ci = 0;
    if (slots <= 2 * kWave)
      merge_parts<T, 2>(lds.part, slots, K, lane, s, ck, ci);
    else if (slots <= 4 * kWave)
      merge_parts<T, 4>(lds.part, slots, K, lane, s, ck, ci);
    else
      merge_parts<T, 8>(lds.part, slots, K, lane, s, ck, ci);
    const uint64_t msk = ballot(ck != 0);
    __builtin_amdgcn_wave_barrier();
    if (ck != 0) s.cand[lanes_below(msk)] = cand_order(ck, ci);
    const int nk = popc(msk);
    __builtin_amdgcn_wave_barrier();
    mine = lane < nk ? s.cand[lane] : 0ull;
    r = lane < nk ? count_above(s.cand, nk, mine) : kWave;
  }
  if (r < K) {
    const int64_t o = row * K + r;
    const uint32_t key = static_cast<uint32_t>(mine >> 32);
    const float v = Traits<T>::from_key(key);
    out.put(out.cand_ids + o, ~static_cast<uint32_t>(mine));
    out.put(out.cand_logit + o, __float_as_uint(v));
    if (out.cand_logprob) out.put(out.cand_logprob + o, __float_as_uint(v - l));
  }
  if (lane == 0 && out.lse) out.put(out.lse + row, __float_as_uint(l));
}


}  // namespace
}  // namespace ubt
