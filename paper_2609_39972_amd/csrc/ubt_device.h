// Device-side building blocks shared by the libubt kernels (gfx950, wave64).
//
//  * order keys: a monotone map from stored logits / scores to unsigned integers, so that
//    "larger value" is "larger key" and -0 == +0.  Key 0 is reserved for "no element".
//  * wave primitives on 64-lane wavefronts: reductions and a ballot-driven radix
//    selection that finds the K-th largest key of 64*R register-resident entries with one
//    compare per entry and bit, the counting done on scalar units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ubt {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float neg_inf() { return -__builtin_huge_valf(); }

// ---- order keys --------------------------------------------------------------------

// bf16 bit pattern -> 16-bit order key (>= 0x7F for every non-NaN value, -inf = 0x7F).
__device__ __forceinline__ uint32_t bf16_key(uint32_t h) {
  h &= 0xFFFFu;
  if ((h & 0x7FFFu) == 0) h = 0;  // -0 -> +0
  return (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
}
__device__ __forceinline__ float bf16_key_value(uint32_t k) {
  const uint32_t h = (k & 0x8000u) ? (k & 0x7FFFu) : (~k & 0xFFFFu);
  return __uint_as_float(h << 16);
}

// fp32 value -> 32-bit order key (>= 0x007FFFFF for every non-NaN value).
__device__ __forceinline__ uint32_t f32_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) == 0) u = 0;  // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float f32_key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// ---- wave helpers ------------------------------------------------------------------

__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

// Number of set bits of `mask` below this lane.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
// Reductions inside aligned groups of 16 lanes.
__device__ __forceinline__ float group16_max(float v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Largest t (over the bits below `nbits`) such that at least `need` of the live entries
// have key >= t, i.e. the need-th largest live key (0 if fewer than `need` are live).
// Entries are key[r] on every lane, r < R; `live[r]` masks entries in or out.
template <int R>
__device__ __forceinline__ uint32_t wave_kth_largest(const uint32_t (&key)[R], const uint64_t (&live)[R],
                                                     int need, int nbits) {
  uint32_t t = 0;
  for (int bit = nbits - 1; bit >= 0; --bit) {
    const uint32_t cand = t | (1u << bit);
    int cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) cnt += popc(ballot(key[r] >= cand) & live[r]);
    if (cnt >= need) t = cand;
  }
  return t;
}

// Selects the `need` largest entries under the order (key desc, sub asc) among the live
// entries of 64*R (key, sub) pairs.  `sub` values are unique among entries with equal
// key.  Returns per row the ballot mask of selected entries.  If fewer than `need`
// entries are live, every live entry is selected.
template <int R>
__device__ __forceinline__ void wave_select(const uint32_t (&key)[R], const uint32_t (&sub)[R],
                                            const uint64_t (&live)[R], int need, int key_bits,
                                            uint64_t (&sel)[R]) {
  int n_live = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) n_live += popc(live[r]);
  if (n_live <= need) {
#pragma unroll
    for (int r = 0; r < R; ++r) sel[r] = live[r];
    return;
  }
  const uint32_t t = wave_kth_largest<R>(key, live, need, key_bits);
  int above = 0, equal = 0;
  uint64_t eq[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    sel[r] = ballot(key[r] > t) & live[r];
    eq[r] = ballot(key[r] == t) & live[r];
    above += popc(sel[r]);
    equal += popc(eq[r]);
  }
  const int rest = need - above;  // 1 <= rest <= equal
  if (rest == equal) {
#pragma unroll
    for (int r = 0; r < R; ++r) sel[r] |= eq[r];
    return;
  }
  // Ties at the threshold: keep the `rest` smallest `sub` values (largest ~sub).
  uint32_t inv[R];
#pragma unroll
  for (int r = 0; r < R; ++r) inv[r] = ~sub[r];
  const uint32_t t2 = wave_kth_largest<R>(inv, eq, rest, 32);
#pragma unroll
  for (int r = 0; r < R; ++r) sel[r] |= ballot(inv[r] >= t2) & eq[r];
}

}  // namespace ubt
