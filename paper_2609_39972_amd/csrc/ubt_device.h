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

// A workgroup barrier ordering LDS only: loads from global memory stay in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }

// Float reductions.  DPP patterns inside a row of 16 lanes: xor 1 and xor 2 within a
// quad, then the mirrors of each half row and of the row; every lane of the row ends
// with the row's result.
template <class Op>
__device__ __forceinline__ float dpp_row_reduce(float v, Op op) {
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false)));
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false)));
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false)));
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false)));
  return v;
}
struct FMax {
  __device__ float operator()(float a, float b) const { return fmaxf(a, b); }
};
struct FAdd {
  __device__ float operator()(float a, float b) const { return a + b; }
};
// Over the wave (every lane active); the result is wave-uniform.
__device__ __forceinline__ float wave_max(float v) {
  v = dpp_row_reduce(v, FMax{});
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}
__device__ __forceinline__ float wave_sum(float v) {
  v = dpp_row_reduce(v, FAdd{});
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}
// Reductions inside aligned groups of 16 lanes.
__device__ __forceinline__ float group16_max(float v) { return dpp_row_reduce(v, FMax{}); }
__device__ __forceinline__ float group16_sum(float v) { return dpp_row_reduce(v, FAdd{}); }

// Lane predicate from a wave mask: the mask is used directly as the lane condition.
__device__ __forceinline__ bool lane_in(uint64_t mask) { return __builtin_amdgcn_inverse_ballot_w64(mask); }

// Max / min of a 32-bit unsigned value over the wave, returned wave-uniform.  Every lane
// must be active: DPP inside rows of 16 lanes, then the four row results on the scalar
// unit.
__device__ __forceinline__ uint32_t dpp_row_umax(uint32_t v) {
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0xB1, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x4E, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x141, 0xF, 0xF, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x140, 0xF, 0xF, false)));
  return v;
}
__device__ __forceinline__ uint32_t dpp_row_umin(uint32_t v) {
  v = min(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0xB1, 0xF, 0xF, false)));
  v = min(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x4E, 0xF, 0xF, false)));
  v = min(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x141, 0xF, 0xF, false)));
  v = min(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x140, 0xF, 0xF, false)));
  return v;
}
// Inclusive prefix sum over the lanes of the wave (lanes 0..l for lane l), by DPP: sums of
// 4, 8 and 16 lanes inside each row of 16, then the rows' totals broadcast into the rows
// after them.  Every lane must be active.
__device__ __forceinline__ uint32_t wave_prefix_sum(uint32_t v) {
  const int x = static_cast<int>(v);
  int s = x + __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);  // row_shr:1
  s += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);         // row_shr:2
  s += __builtin_amdgcn_update_dpp(0, x, 0x113, 0xF, 0xF, true);         // row_shr:3
  s += __builtin_amdgcn_update_dpp(0, s, 0x114, 0xF, 0xE, false);        // row_shr:4, lanes 4..15
  s += __builtin_amdgcn_update_dpp(0, s, 0x118, 0xF, 0xC, false);        // row_shr:8, lanes 8..15
  s += __builtin_amdgcn_update_dpp(0, s, 0x142, 0xA, 0xF, false);        // row_bcast:15, rows 1, 3
  s += __builtin_amdgcn_update_dpp(0, s, 0x143, 0xC, 0xF, false);        // row_bcast:31, rows 2, 3
  return static_cast<uint32_t>(s);
}

// Sum over each quad of lanes (every lane of the quad gets it).
__device__ __forceinline__ int quad_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  return v;
}
__device__ __forceinline__ uint32_t wave_umax(uint32_t v) {
  v = dpp_row_umax(v);
  const uint32_t a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
  const uint32_t c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
  return max(max(a, b), max(c, d));
}
__device__ __forceinline__ uint32_t wave_umin(uint32_t v) {
  v = dpp_row_umin(v);
  const uint32_t a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
  const uint32_t c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
  return min(min(a, b), min(c, d));
}

// Largest and smallest live key (0 and ~0 when none is live).
template <int R>
__device__ __forceinline__ void live_key_range(const uint32_t (&key)[R], const uint64_t (&live)[R], uint32_t& kmax,
                                               uint32_t& kmin) {
  uint32_t hi = 0u, lo = ~0u;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const bool l = lane_in(live[r]);
    hi = max(hi, l ? key[r] : 0u);
    lo = min(lo, l ? key[r] : ~0u);
  }
  kmax = wave_umax(hi);
  kmin = wave_umin(lo);
}

// The next bit of a radix search over keys: m >> 1, or 0 (the search is over) when
// need <= cnt <= need + span.  One scalar compare and select, so that the loop that
// calls it ends on a single test of the returned value; cnt, need and span must be
// wave-uniform.
__device__ __forceinline__ uint32_t radix_next(uint32_t m, int cnt, int need, uint32_t span) {
  uint32_t next = __builtin_amdgcn_readfirstlane(m >> 1), d;
  asm volatile("s_sub_u32 %1, %2, %3\n\ts_cmp_gt_u32 %1, %4\n\ts_cselect_b32 %0, %0, 0"
               : "+s"(next), "=&s"(d)
               : "s"(__builtin_amdgcn_readfirstlane(cnt)), "s"(__builtin_amdgcn_readfirstlane(need)),
                 "s"(__builtin_amdgcn_readfirstlane(span))
               : "scc");
  return next;
}

// Radix search for the need-th largest live key, for need < the number of live keys.
// Live keys share the bits above the highest bit where the largest and the smallest of
// them differ, so the search starts below that common prefix.  Returns true, with sel =
// the live entries with key >= s, at the first s that splits off exactly `need` of them;
// otherwise returns false with t = the need-th largest key (then more than `need` keys
// are >= t: the boundary is a tie).
template <int R>
__device__ __forceinline__ bool radix_split(const uint32_t (&key)[R], const uint64_t (&live)[R], int need,
                                            uint64_t (&sel)[R], uint32_t& t) {
  uint32_t kmax, kmin;
  live_key_range<R>(key, live, kmax, kmin);
  t = kmax;
  if (kmax == kmin) return false;
  uint32_t m = 0x80000000u >> __clz(kmax ^ kmin);
  t = kmax & ~(m | (m - 1u));
  int cnt;
  do {
    const uint32_t cand = t | m;
    cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      sel[r] = ballot(key[r] >= cand) & live[r];
      cnt += popc(sel[r]);
    }
    t = cnt > need ? cand : t;
    m = radix_next(m, cnt, need, 0u);
  } while (m != 0u);
  return cnt == need;
}

// A threshold t with at least `need` live keys >= t, refined only until at most `cap` of
// them are (cap >= need); 0 if fewer than `need` are live.  Cheaper than the exact
// need-th largest key when a slightly lower bound will do.
template <int R>
__device__ __forceinline__ uint32_t wave_threshold(const uint32_t (&key)[R], const uint64_t (&live)[R], int need,
                                                   int cap) {
  int n_live = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) n_live += popc(live[r]);
  if (n_live < need) return 0u;
  uint32_t kmax, kmin;
  live_key_range<R>(key, live, kmax, kmin);
  if (n_live <= cap || kmax == kmin) return kmin;
  uint32_t m = 0x80000000u >> __clz(kmax ^ kmin);
  uint32_t t = kmax & ~(m | (m - 1u));
  do {
    const uint32_t cand = t | m;
    int cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) cnt += popc(ballot(key[r] >= cand) & live[r]);
    t = cnt >= need ? cand : t;
    m = radix_next(m, cnt, need, static_cast<uint32_t>(cap - need));
  } while (m != 0u);
  return t;
}

// Selects the `need` largest entries under the order (key desc, sub asc) among the live
// entries of 64*R (key, sub) pairs.  `sub` values are unique among entries with equal
// key.  Returns per row the ballot mask of selected entries.  If fewer than `need`
// entries are live, every live entry is selected.  Every lane must be active.
template <int R>
__device__ __forceinline__ void wave_select(const uint32_t (&key)[R], const uint32_t (&sub)[R],
                                            const uint64_t (&live)[R], int need, int key_bits,
                                            uint64_t (&sel)[R]) {
  (void)key_bits;
  int n_live = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) n_live += popc(live[r]);
  if (n_live <= need) {
#pragma unroll
    for (int r = 0; r < R; ++r) sel[r] = live[r];
    return;
  }
  uint32_t t;
  if (radix_split<R>(key, live, need, sel, t)) return;
  int above = 0;
  uint64_t eq[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    sel[r] = ballot(key[r] > t) & live[r];
    eq[r] = ballot(key[r] == t) & live[r];
    above += popc(sel[r]);
  }
  // Ties at the threshold: keep the `rest` smallest `sub` values (largest ~sub).
  const int rest = need - above;  // 1 <= rest < entries tied at t
  uint32_t inv[R];
#pragma unroll
  for (int r = 0; r < R; ++r) inv[r] = ~sub[r];
  uint64_t tie[R];
  uint32_t u;
  if (!radix_split<R>(inv, eq, rest, tie, u)) {
#pragma unroll
    for (int r = 0; r < R; ++r) tie[r] = ballot(inv[r] >= u) & eq[r];
  }
#pragma unroll
  for (int r = 0; r < R; ++r) sel[r] |= tie[r];
}

}  // namespace ubt
