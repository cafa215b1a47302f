// The whole draft step as two launches: softmax statistics and top-K candidates over the
// vocabulary, the selector scores, and the tree search with its ancestor mask.
//
// Method / Unigram Proposer, Eq. (ubtree-unigram) and "Candidate Sets" (per-position LSE
// and C_i); Method / Parallel Computation, Eq. (ubtree-edge-matrix), Depth Calibration,
// Eq. (ubtree-depth), and Appendix A / Path Scores, Eq. (ubtree-path) (log q^bi);
// Appendix A, Algorithm 1 with Eqs. (ubtree-frontier) and (ubtree-pruning) (the tree);
// Appendix A / Verification via Tree-attention (the mask).
//
// The sweep is bound by HBM bandwidth and the search of one sequence is a long chain of
// dependent steps on one wave, and the search of depth d needs only the rows of
// positions up to d.  So the rows are swept in two parts:
//   * the head launch sweeps positions 0..d1-1 of every sequence, one row per workgroup
//     of 8 waves, as the top-K kernel does;
//   * the tail launch sweeps positions d1..gamma-1 the same way while one searcher
//     workgroup per sequence (the lowest workgroup indices, so they are dispatched
//     first) computes the score slabs of the head positions and searches them.  A tail
//     row publishes its candidates with device-coherent stores and a flag; the searcher
//     takes each tail position as soon as its flag is up, and finishes the search.
// d1 is about half of gamma, and small enough that the tail's row workgroups and the
// searchers take at most one compute unit each.  (Measured at B = 32, gamma = 15: d1 = 8
// beat every other split from 6 to 12, and 8-wave workgroups beat 16-wave ones in both
// launches.)  Each row's results are those of ubt_topk, and the
// slabs and the search are the code of ubt_draft_tree, so every output is that of the
// two separate calls (LSE and log-probs in the same order too).
//
// Row workers never wait; searcher waves wait only on flags that tail rows of the same
// launch set unconditionally, each wait bounded in time.  The flags are reset by the
// searcher that read them, leaving the workspace ready for the next call.
#include "bigram_tile.h"
#include "search.h"
#include "sweep.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

constexpr int kRowWaves = kWaves;  // waves per workgroup of both launches (8)
constexpr uint64_t kWaitTicks = 100000000ull;  // 1 s of the 100 MHz real-time counter
constexpr uint32_t kFlagBase = 256;            // byte offset of the row flags in the workspace

__device__ __forceinline__ void store_agent32(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t load_agent32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Waits until every memory operation issued so far by this wave has completed.
__device__ __forceinline__ void wait_all_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

struct RowArgs {
  const void* logits;
  int64_t V, stride_b, stride_i;
  int B, gamma, K;
  int d1;  // positions 0..d1-1 belong to the head launch
  int32_t* cand_ids;
  float* cand_logit;
  float* cand_logprob;
  float* lse;
  uint32_t* err;   // set when a searcher wait timed out
  uint32_t* flag;  // [B * gamma] 1 once a tail row's candidates are out
};

// Sweeps output row (b, i) with the workgroup's kRowWaves waves.
template <typename T, bool kCoherent>
__device__ __forceinline__ void sweep_one(const RowArgs& p, RowLdsT<kRowWaves>& lds, int b, int i) {
  const int64_t orow = static_cast<int64_t>(b) * p.gamma + i;
  const T* rp = static_cast<const T*>(p.logits) + b * p.stride_b + i * p.stride_i;
  sweep_row<T, true, kRowWaves>(lds, rp, p.V, p.K, orow,
                                RowOut{p.cand_ids, p.cand_logit, p.cand_logprob, p.lse, kCoherent});
}

// Head launch: positions 0..d1-1 of every sequence, one row per workgroup.
template <typename T>
__global__ __launch_bounds__(kRowWaves* kWave, 4) void head_rows_kernel(RowArgs p) {
  __shared__ RowLdsT<kRowWaves> lds;
  const int r = static_cast<int>(blockIdx.x);
  sweep_one<T, false>(p, lds, r % p.B, r / p.B);
}

// Spins until *f is set; false if the wait ran out of time.
__device__ __forceinline__ bool wait_flag(const uint32_t* f, uint64_t t0) {
  for (;;) {
    if (__builtin_amdgcn_readfirstlane(load_agent32(f)) != 0u) return true;
    if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) return false;
    __builtin_amdgcn_s_sleep(4);
  }
}

struct SearcherLayout {
  FastLayout fast;
  uint32_t clogit, rready, total;
};

__host__ __device__ inline SearcherLayout searcher_layout(int gamma, int K, int W) {
  SearcherLayout L{};
  L.fast = fast_layout(gamma, K, W);
  uint32_t q = L.fast.total;
  L.clogit = q;
  q += static_cast<uint32_t>((gamma * K * sizeof(float) + 15) & ~static_cast<size_t>(15));
  L.rready = q;
  q += static_cast<uint32_t>((gamma * sizeof(uint32_t) + 15) & ~static_cast<size_t>(15));
  L.total = q;
  return L;
}

// One sequence's selector slabs and tree search.  Wave 0 searches; waves 1.. take the
// positions round-robin: they bring the position's candidates into LDS (a head row from
// memory written by the head launch; a tail row once its flag is up, with device-coherent
// loads), compute its slab once the predecessor position's candidates are in, and
// publish it to the search wave.
template <int KT, int R>
__device__ __forceinline__ void searcher(const RowArgs& p, const TreeArgs& a, const SelectorArgs& s, uint64_t magic_w,
                                         unsigned char* smem, int w, int nw, int lane) {
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
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  for (int i = w - 1; i < gamma; i += nw - 1) {
    const int64_t bi = static_cast<int64_t>(b) * gamma + i;
    if (i < p.d1) {
      if (lane < KT) {
        sm.cids[i * KT + lane] = p.cand_ids[bi * KT + lane];
        clogit[i * KT + lane] = p.cand_logit[bi * KT + lane];
      }
    } else {
      if (!wait_flag(&p.flag[bi], t0) && lane == 0) store_agent32(p.err, 1u);
      if (lane < KT) {
        sm.cids[i * KT + lane] = static_cast<int32_t>(load_agent32(reinterpret_cast<const uint32_t*>(p.cand_ids) +
                                                                   bi * KT + lane));
        clogit[i * KT + lane] =
            __uint_as_float(load_agent32(reinterpret_cast<const uint32_t*>(p.cand_logit) + bi * KT + lane));
      }
      if (lane == 0) store_agent32(&p.flag[bi], 0u);  // read: ready for the next call
    }
    publish_slab(rready, i);
    if (i > 0) wait_slab(rready, i - 1);
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

// Tail launch: workgroups 0..B-1 search; the others sweep positions d1..gamma-1
// (depth-major) and raise each row's flag once its candidates have completed.
template <typename T, int KT, int R>
__global__ __launch_bounds__(kRowWaves* kWave, 4) void draft_tail_kernel(RowArgs p, TreeArgs a, SelectorArgs s,
                                                                          uint64_t magic_w) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int nw = static_cast<int>(blockDim.x) / kWave;
  if (static_cast<int>(blockIdx.x) < p.B) {
    searcher<KT, R>(p, a, s, magic_w, smem_raw, w, nw, lane);
    return;
  }
  const int r = static_cast<int>(blockIdx.x) - p.B;
  const int b = r % p.B, i = p.d1 + r / p.B;
  sweep_one<T, true>(p, *reinterpret_cast<RowLdsT<kRowWaves>*>(smem_raw), b, i);
  // Wave 0 wrote the row's results (device-coherent stores); once they have completed,
  // the flag goes up.
  if (w == 0) {
    wait_all_memory();
    if (lane == 0) store_agent32(&p.flag[static_cast<int64_t>(b) * p.gamma + i], 1u);
  }
}

int compute_units() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

}  // namespace

// ---- host side ------------------------------------------------------------------------------
size_t step_workspace_bytes(int B, int gamma) {
  return kFlagBase + static_cast<size_t>(B) * gamma * sizeof(uint32_t);
}

// Positions 0..d1-1 go to the head launch: at least half of them, and few enough that
// the tail's rows and the searchers take at most one workgroup per compute unit.  0 if no
// such split exists.
int step_split(int B, int gamma) {
  const int cus = compute_units();
  if (gamma < 2 || cus <= 0 || B >= cus) return 0;
  int d1 = (gamma + 1) / 2;
  const int tail_max = (cus - B) / B;  // tail positions that fit beside the searchers
  if (gamma - d1 > tail_max) d1 = gamma - tail_max;
  return d1 < gamma ? d1 : 0;
}

bool draft_step_fused(int dtype, bool aligned, int B, int gamma, int64_t V, int K, int feat_dtype, int W) {
  if (!aligned || feat_dtype != 1 || B > kMaxStepSequences) return false;
  if (!draft_tree_fused(feat_dtype, gamma, K, W)) return false;
  (void)dtype;
  (void)V;
  return step_split(B, gamma) > 0;
}

hipError_t launch_draft_step(const void* logits, int dtype, int B, int gamma, int64_t V, int64_t stride_b,
                             int64_t stride_i, int K, int32_t* cand_ids, float* cand_logit, float* cand_logprob,
                             float* lse, const SelectorArgs& s, const TreeArgs& a, void* workspace,
                             hipStream_t stream) {
  RowArgs p{};
  p.logits = logits;
  p.V = V;
  p.stride_b = stride_b;
  p.stride_i = stride_i;
  p.B = B;
  p.gamma = gamma;
  p.K = K;
  p.d1 = step_split(B, gamma);
  p.cand_ids = cand_ids;
  p.cand_logit = cand_logit;
  p.cand_logprob = cand_logprob;
  p.lse = lse;
  char* ws = static_cast<char*>(workspace);
  p.err = reinterpret_cast<uint32_t*>(ws);
  p.flag = reinterpret_cast<uint32_t*>(ws + kFlagBase);

  const dim3 block(kRowWaves * kWave);
  if (dtype == 1)
    hipLaunchKernelGGL(head_rows_kernel<uint16_t>, dim3(static_cast<unsigned>(B * p.d1)), block, 0, stream, p);
  else
    hipLaunchKernelGGL(head_rows_kernel<float>, dim3(static_cast<unsigned>(B * p.d1)), block, 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  const uint64_t magic_w = (0x100000000ull + a.W - 1) / a.W;
  const size_t row_smem = sizeof(RowLdsT<kRowWaves>);
  const size_t search_smem = searcher_layout(gamma, K, a.W).total;
  const size_t smem = row_smem > search_smem ? row_smem : search_smem;
  const dim3 grid(static_cast<unsigned>(B + B * (gamma - p.d1)));
  const int wk = a.W * K;
#define UBT_TAIL_LAUNCH(TT, KK, RR)                                                                         \
  do {                                                                                                      \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&draft_tail_kernel<TT, KK, RR>),               \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));          \
    hipLaunchKernelGGL((draft_tail_kernel<TT, KK, RR>), grid, block, smem, stream, p, a, s, magic_w);      \
  } while (0)
#define UBT_TAIL_ROWS(TT, KK)       \
  do {                              \
    if (wk <= 64)                   \
      UBT_TAIL_LAUNCH(TT, KK, 1);   \
    else if (wk <= 128)             \
      UBT_TAIL_LAUNCH(TT, KK, 2);   \
    else if (wk <= 256)             \
      UBT_TAIL_LAUNCH(TT, KK, 4);   \
    else if (wk <= 384)             \
      UBT_TAIL_LAUNCH(TT, KK, 6);   \
    else                            \
      UBT_TAIL_LAUNCH(TT, KK, 8);   \
  } while (0)
#define UBT_TAIL_K(TT)         \
  do {                         \
    if (K == 4)                \
      UBT_TAIL_ROWS(TT, 4);    \
    else if (K == 8)           \
      UBT_TAIL_ROWS(TT, 8);    \
    else                       \
      UBT_TAIL_ROWS(TT, 16);   \
  } while (0)
  if (dtype == 1)
    UBT_TAIL_K(uint16_t);
  else
    UBT_TAIL_K(float);
#undef UBT_TAIL_K
#undef UBT_TAIL_ROWS
#undef UBT_TAIL_LAUNCH
  return hipGetLastError();
}

}  // namespace ubt
