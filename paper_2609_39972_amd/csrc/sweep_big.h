// Top-K candidates of one logit row for large K (K > 16), one workgroup of 8 waves: the
// streaming pass of sweep.h with a larger candidate buffer, then an exact selection over
// all the waves' candidates at once.
//
// Method / Unigram Proposer, Eq. (ubtree-unigram), q_i = softmax(u_i), and "Candidate
// Sets": C_i = the K tokens of largest q_i, ranked on the logits with ties to the lower
// token id.
//
// With K = 64 a first threshold taken from one tile per wave lets several hundred elements
// of the row through; a per-wave top K merged by one wave would cost several radix
// selections at the end of the row.  Here every wave keeps its passing groups (up to
// kBigCap of them; a fuller buffer still merges into a running top K as in sweep.h), and
// the whole workgroup selects the K largest order values (key desc, id asc) among all the
// candidates by a most-significant-digit radix descent: per pass one LDS histogram of 256
// bins over the candidates that share the prefix fixed so far, one barrier, and every wave
// finds the bin holding the K-th value from the same counts.  The descent stops at the
// first bin that closes the count exactly (usually after the key bits); the K selected
// values are then ranked by counting and written in order.
#pragma once

#include "sweep.h"

namespace ubt {
namespace {

constexpr int kBigCap = 192;     // candidate groups per wave
constexpr int kKeyPasses = 4;    // digits of a 32-bit key
constexpr int kIdPasses = 4;     // digits of a 32-bit id
constexpr int kFinCap = 512;     // candidates ranked at the end
constexpr int kCandRegs = 4;     // a wave's candidates held in registers (64 each)

struct BigRowLds {
  WaveLdsT<kBigCap> wave[kWaves];
  uint32_t lane_max[kWaves * kWave];
  uint32_t hist[kKeyPasses + kIdPasses][256];  // one histogram per pass
  uint64_t fin[kFinCap + 16];                   // the candidates ranked at the end, unordered
  float2 ms[kWaves];                            // each wave's (max, sum)
  uint32_t wthr[kWaves];                        // each wave's threshold key: a lower bound of the row's K-th
  uint32_t wtop[kWaves];                        // each wave's largest candidate key
  uint2 wc[kWaves][kCandRegs * kWave];          // each wave's candidates (key, id), staged
  uint32_t nfin;
};

// One step of a radix descent, run by a whole wave on a 256-bin histogram h of the values
// at the current prefix: the digit d* whose bin holds the need-th largest value, i.e.
// count(bins > d*) < need <= count(bins >= d*).  Returns d* and sets `above` to
// count(bins > d*) and `in_bin` to the count of bin d*.  Lane l holds bins 252 - 4 l ..
// 255 - 4 l, so a prefix sum over the lanes counts the bins from the top.
__device__ __forceinline__ uint32_t descend(const uint32_t* h, int need, int lane, int& above, int& in_bin) {
  const int base = 4 * (kWave - 1 - lane);
  const uint4 hv = reinterpret_cast<const uint4*>(h)[kWave - 1 - lane];  // bins base .. base + 3
  const uint32_t own = hv.x + hv.y + hv.z + hv.w;
  const uint32_t s4 = wave_prefix_sum(own) - own;  // bins above this lane's
  const uint32_t s3 = s4 + hv.w, s2 = s3 + hv.z, s1 = s2 + hv.y, s0 = s1 + hv.x;
  const uint32_t nd = static_cast<uint32_t>(need);
  const int dig = s3 >= nd ? 3 : (s2 >= nd ? 2 : (s1 >= nd ? 1 : 0));
  const uint32_t cnt = dig == 3 ? hv.w : (dig == 2 ? hv.z : (dig == 1 ? hv.y : hv.x));
  const uint32_t abv = dig == 3 ? s4 : (dig == 2 ? s3 : (dig == 1 ? s2 : s1));
  // Exactly one lane has s0 >= need > s4 (the values at the prefix number at least need).
  const uint64_t at = ballot(s0 >= nd && s4 < nd);
  const int src = at != 0ull ? static_cast<int>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(__builtin_ctzll(at)))) : 0;
  above = static_cast<int>(__builtin_amdgcn_readlane(abv, src));
  in_bin = static_cast<int>(__builtin_amdgcn_readlane(cnt, src));
  return __builtin_amdgcn_readlane(static_cast<uint32_t>(base + dig), src);
}

// The row at rp (V >= K elements) of global row index `row`, K <= 64.  Writes
// cand_*[row * K, row * K + K) and lse[row].
template <typename T, bool kAligned>
__device__ __forceinline__ void sweep_row_big(BigRowLds& lds, const T* __restrict__ rp, int64_t V, int K, int64_t row,
                                              const RowOut& out) {
  constexpr int EPG = Traits<T>::kPer;
  const int nw = blockDim.x / kWave;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const __amdgpu_buffer_rsrc_t rsrc = row_resource(rp, static_cast<uint32_t>(V * static_cast<int64_t>(sizeof(T))));
  auto& s = lds.wave[w];
  for (int e = static_cast<int>(threadIdx.x); e < (kKeyPasses + kIdPasses) * 256; e += static_cast<int>(blockDim.x))
    (&lds.hist[0][0])[e] = 0u;
  if (threadIdx.x == 0) lds.nfin = 0u;  // published by the barrier inside the pass
  WaveState st;
  stream_row<T, kAligned, kWaves, true>(s, lds.lane_max, rp, V, K, nw, w, lane, rsrc, st);

  // Candidates of this wave: the buffered elements that pass its threshold (strictly once
  // it holds a running top K: later elements carry larger ids) and, if it merged, its
  // running top K; every candidate must also reach `tall`, the best threshold of any wave
  // (0 while the waves' thresholds are not yet shared).  each_buffered calls fn(key, id,
  // live) for them per lane, from the buffer.
  const int tot = st.nbuf * EPG;
  uint32_t tall = 0u;
  auto each_buffered = [&](auto&& fn) {
    for (int e0 = 0; e0 < tot; e0 += kWave) {
      const int e = e0 + lane;
      uint32_t k = 0u, id = 0u;
      bool live = false;
      if (e < tot) {
        const int g = e / EPG, j = e % EPG;
        const uint32_t word = reinterpret_cast<const uint32_t*>(&s.data[g])[j * 4 / EPG];
        const uint32_t bits = EPG == 8 ? (word >> (16 * (j & 1))) & 0xFFFFu : word;
        const int64_t gid = static_cast<int64_t>(s.base[g]) + j;
        if (gid < V) {
          k = Traits<T>::key_bits(bits);
          id = static_cast<uint32_t>(gid);
          live = (st.strict ? k > st.thr : k >= st.thr) && k >= tall;
        }
      }
      fn(k, id, live);
    }
    if (st.merged) fn(st.cur_key, st.cur_id, lane < K && st.cur_key != 0u && st.cur_key >= tall);
  };
  // One pass over the buffer, a group per lane, stages the candidates (each lane's at
  // its offset from a prefix sum of the counts); up to kCandRegs * 64 of them then live in
  // registers (ck, ci, held by lanes with cl) for the passes below.
  uint2* wc = lds.wc[w];
  int nc = 0;
  uint32_t top = 0u;
  for (int g0 = 0; g0 < st.nbuf; g0 += kWave) {
    const int g = g0 + lane;
    uint32_t km[EPG];
    uint32_t live = 0u, gbase = 0u;
    if (g < st.nbuf) {
      const u32x4 v = s.data[g];
      gbase = s.base[g];
#pragma unroll
      for (int j = 0; j < EPG; ++j) {
        const uint32_t word = v[j * 4 / EPG];
        const uint32_t bits = EPG == 8 ? (word >> (16 * (j & 1))) & 0xFFFFu : word;
        km[j] = Traits<T>::key_bits(bits);
        const bool in = static_cast<int64_t>(gbase) + j < V && (st.strict ? km[j] > st.thr : km[j] >= st.thr);
        live |= in ? 1u << j : 0u;
        top = max(top, in ? km[j] : 0u);
      }
    }
    const uint32_t cnt = static_cast<uint32_t>(__builtin_popcount(live));
    const uint32_t incl = wave_prefix_sum(cnt);
    int pos = nc + static_cast<int>(incl - cnt);
#pragma unroll
    for (int j = 0; j < EPG; ++j) {
      if ((live >> j) & 1u) {
        if (pos < kCandRegs * kWave) wc[pos] = make_uint2(km[j], gbase + j);
        ++pos;
      }
    }
    nc += static_cast<int>(__builtin_amdgcn_readlane(incl, kWave - 1));
  }
  if (st.merged) {
    const bool in = lane < K && st.cur_key != 0u;
    const uint64_t m = ballot(in);
    const int pos = nc + static_cast<int>(lanes_below(m));
    if (in && pos < kCandRegs * kWave) wc[pos] = make_uint2(st.cur_key, st.cur_id);
    nc += popc(m);
    top = max(top, in ? st.cur_key : 0u);
  }
  const bool in_regs = nc <= kCandRegs * kWave;
  __builtin_amdgcn_wave_barrier();
  uint32_t ck[kCandRegs], ci[kCandRegs];
  bool cl[kCandRegs];
#pragma unroll
  for (int r = 0; r < kCandRegs; ++r) {
    const int e = r * kWave + lane;
    const uint2 v = wc[e];
    cl[r] = in_regs && e < nc;
    ck[r] = v.x;
    ci[r] = v.y;
  }
  auto each = [&](auto&& fn) {
    if (in_regs) {
#pragma unroll
      for (int r = 0; r < kCandRegs; ++r) fn(ck[r], ci[r], cl[r] && ck[r] >= tall);
    } else {
      each_buffered(fn);
    }
  };
  top = wave_umax(top);
  const float wm = wave_max(st.lm);
  const float wsum = wave_sum((st.lm == neg_inf()) ? 0.f : st.ls * fast_exp2((st.lm - wm) * kLog2e));
  if (lane == 0) {
    lds.ms[w] = make_float2(wm, wsum);
    lds.wthr[w] = st.thr;
    lds.wtop[w] = top;
  }
  __syncthreads();
  uint32_t ktop = 0u;
  for (int j = 0; j < nw; ++j) {
    tall = max(tall, lds.wthr[j]);
    ktop = max(ktop, lds.wtop[j]);
  }

  // Radix descent over the key bits below the common prefix of [tall, ktop] (every
  // candidate key lies there), 8 bits a pass: kstar = the K-th largest candidate key,
  // with `need` candidates of key kstar among the K and `n_eq` candidates of that key.
  int need = K, pass = 0, n_eq = 0;
  uint32_t kstar = ktop;
  {
    int shift = 32 - __builtin_clz(tall ^ ktop | 1u);  // bits [shift, 32) are common
    if (tall == ktop) shift = 0;
    uint32_t prefix = shift >= 32 ? 0u : ktop >> shift;
    int above = 0, in_bin = 0;
    if (shift == 0) {
      // One key: count it.
      uint32_t* h = lds.hist[0];
      each([&](uint32_t k, uint32_t, bool live) {
        const uint64_t m = ballot(live);
        if (m != 0ull && lane == 0) atomicAdd(&h[0], static_cast<uint32_t>(popc(m)));
      });
      __syncthreads();
      n_eq = static_cast<int>(h[0]);
      pass = 1;
    }
    while (shift > 0) {
      const int wd = shift < 8 ? shift : 8;
      shift -= wd;
      uint32_t* h = lds.hist[pass++];
      const uint32_t dmask = (1u << wd) - 1u;
      each([&](uint32_t k, uint32_t, bool live) {
        if (live && (shift + wd >= 32 ? 0u : k >> (shift + wd)) == prefix) atomicAdd(&h[(k >> shift) & dmask], 1u);
      });
      __syncthreads();
      const uint32_t d = descend(h, need, lane, above, in_bin);
      need -= above;
      prefix = (prefix << wd) | d;
      n_eq = in_bin;
    }
    kstar = prefix;
  }
  // The candidates with key > kstar (K - need of them) are in.  Of the n_eq with key
  // kstar the need of smallest id are: with n_eq == need all of them; with few enough,
  // they all go to the final ranking; otherwise a radix descent over ~id picks them.
  uint32_t id_cut = 0u;  // key-kstar candidates need ~id >= id_cut
  if (n_eq != need && (K - need) + n_eq > kFinCap) {
    int shift = 32;
    uint32_t prefix = 0u;
    int above = 0, in_bin = 0;
    while (shift > 0) {
      shift -= 8;
      uint32_t* h = lds.hist[pass++];
      each([&](uint32_t k, uint32_t id, bool live) {
        const uint32_t x = ~id;
        if (live && k == kstar && (shift + 8 >= 32 ? 0u : x >> (shift + 8)) == prefix) atomicAdd(&h[(x >> shift) & 0xFFu], 1u);
      });
      __syncthreads();
      const uint32_t d = descend(h, need, lane, above, in_bin);
      need -= above;
      prefix = (prefix << 8) | d;
      if (in_bin == need) {
        id_cut = prefix << shift;
        break;
      }
    }
    if (shift == 0) id_cut = prefix;
  }
  // Gather every candidate with key > kstar, or key == kstar and ~id >= id_cut, rank each
  // among them by counting and write the first K in order.
  each([&](uint32_t k, uint32_t id, bool live) {
    const bool pick = live && (k > kstar || (k == kstar && ~id >= id_cut));
    const uint64_t m = ballot(pick);
    if (m == 0ull) return;
    uint32_t o = 0u;
    if (lane == 0) o = atomicAdd(&lds.nfin, static_cast<uint32_t>(popc(m)));
    const int pos = static_cast<int>(__builtin_amdgcn_readlane(o, 0)) + static_cast<int>(lanes_below(m));
    if (pick) lds.fin[pos] = cand_order(k, id);
  });
  __syncthreads();
  const int nfin = static_cast<int>(lds.nfin);

  float m = neg_inf();
  for (int j = 0; j < nw; ++j) m = fmaxf(m, lds.ms[j].x);
  float e = 0.f;
  for (int j = 0; j < nw; ++j) {
    const float2 msj = lds.ms[j];
    if (msj.x != neg_inf()) e += msj.y * fast_exp2((msj.x - m) * kLog2e);
  }
  const float l = (m == neg_inf()) ? neg_inf() : m + fast_log2(e) * kLn2;
  // Entry t is ranked by the quad of lanes 4 (t % 16) .. + 3 of wave (t / 16) % nw: lane q
  // of the quad counts the entries ahead of it among fin[k], k = q mod 4.
  const int q = lane & 3;
  for (int t0 = 16 * w; t0 < nfin; t0 += 16 * nw) {
    const int t = t0 + (lane >> 2);
    const uint64_t mine = t < nfin ? lds.fin[t] : 0ull;
    int ahead[4] = {0, 0, 0, 0};
    for (int k0 = 0; k0 < nfin; k0 += 16) {
      uint64_t o[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) o[u] = lds.fin[k0 + 4 * u + q];
#pragma unroll
      for (int u = 0; u < 4; ++u) ahead[u] += (k0 + 4 * u + q < nfin && o[u] > mine) ? 1 : 0;
    }
    const int r = t < nfin ? quad_sum((ahead[0] + ahead[1]) + (ahead[2] + ahead[3])) : kFinCap;
    if (q == 0 && r < K) {
      const int64_t o = row * K + r;
      const float v = Traits<T>::from_key(static_cast<uint32_t>(mine >> 32));
      out.put(out.cand_ids + o, ~static_cast<uint32_t>(mine));
      out.put(out.cand_logit + o, __float_as_uint(v));
      if (out.cand_logprob) out.put(out.cand_logprob + o, __float_as_uint(v - l));
    }
  }
  if (threadIdx.x == 0 && out.lse) out.put(out.lse + row, __float_as_uint(l));
}

}  // namespace
}  // namespace ubt
