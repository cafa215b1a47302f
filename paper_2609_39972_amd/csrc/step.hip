// The whole draft step in one launch: softmax statistics and top-K candidates over the
// vocabulary, the selector scores, and the tree search with its ancestor mask.
//
// Method / Unigram Proposer, Eq. (ubtree-unigram) and "Candidate Sets" (per-position LSE
// and C_i); Method / Parallel Computation, Eq. (ubtree-edge-matrix), Depth Calibration,
// Eq. (ubtree-depth), and Appendix A / Path Scores, Eq. (ubtree-path) (log q^bi);
// Appendix A, Algorithm 1 with Eqs. (ubtree-frontier) and (ubtree-pruning) (the tree);
// Appendix A / Verification via Tree-attention (the mask).
//
// The sweep is bound by HBM bandwidth; the search of one sequence is a long chain of
// dependent steps on one wave, and its depth d needs only the rows of positions up to d.
// If every row is swept by its own workgroup, all rows finish together near the end of
// the sweep and the search can only start then.  Here the rows are swept in depth order
// instead, each row cut into C chunks of whole tiles, so the early positions come out
// first and the search runs while the later ones are swept:
//   * workgroups 0..B-1 are the searchers, one per sequence (the lowest indices, so they
//     are dispatched first).  Their helper waves merge a row's C chunk results into its
//     LSE and sorted top K as soon as the last chunk is in, compute that position's score
//     slab, and publish it to wave 0, which runs the search;
//   * workgroup B + t sweeps work item t: chunk t % C of sequence (t / C) % B at position
//     t / (B C).  Workgroups are dispatched in index order as earlier ones retire, so the
//     items run depth-major with a window of resident items (two workgroups per compute
//     unit: at B = 32, C = 2 about eight positions in flight, the first rows ready after
//     about 12 of 31 us of sweep).  An item runs the one-row sweep on its chunk, writes the
//     chunk's LSE and top K (ids relative to the chunk) with device-coherent stores, waits for
//     them to complete, and adds 1 to the row's counter.
// The hand-over between workgroups (which may sit on different XCDs, each with its own
// L2) uses agent-scope atomics only: the chunk results are written with relaxed
// agent-scope atomic stores and read with relaxed agent-scope atomic loads, so they go to
// and come from the device-coherent level and no L2 holds a stale copy.  The ordering is
// the hardware's: the producer's wave waits for its stores to be acknowledged
// (s_waitcnt 0) before it issues the counter increment, and a helper issues its loads of
// the results only after its counter load has returned the final count.  A release on
// the increment and an acquire after the wait express the same order in the language's
// memory model, but at agent scope they compile to an L2 write-back per chunk and an L2
// invalidation per row: measured 71.3 us per call against 45.2 us at B = 32, V = 151936.
// The merge of the chunks is exact for the candidates (a selection on the same order
// values) and sums the chunks' exponentials in chunk order, so the candidates, the slabs
// and the tree are those of ubt_topk followed by ubt_draft_tree, and LSE and log-probs
// agree with them to fp32 rounding.
//
// Sweep workgroups never wait.  Searcher waves wait only on counters that sweep
// workgroups of the same launch raise unconditionally, each wait bounded in time; the
// searcher that read a counter resets it, leaving the workspace ready for the next call.
#include <mutex>

#include "bigram_tile.h"
#include "pipe_search.h"
#include "search.h"
#include "sweep.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

// Waves per workgroup, and chunks per row (C K <= 64 as well).  Measured at B = 32,
// gamma = 15, V = 151936, K = 8: C = 2 gave 45.4 us per call; C = 1 50.7 us (every row
// finishes near the end of the sweep), C = 4 53 us and C = 8 75 us (each item is too
// short to cover its own load latency and merge); 4-wave workgroups with C = 4 48.8 us.
constexpr int kPipeWaves = 8;
constexpr int kPipeMaxChunks = 2;
constexpr uint32_t kCountBase = 256;           // byte offset of the row counters in the workspace

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

struct PipeArgs {
  const void* logits;
  int64_t V, stride_b, stride_i;
  int B, gamma, K;
  int chunks;         // C: chunks per row
  int64_t chunk_len;  // elements per chunk, a whole number of tiles; the last chunk is shorter
  int32_t* cand_ids;
  float* cand_logit;
  float* cand_logprob;
  float* lse;
  uint32_t* err;      // set when a searcher wait timed out
  uint32_t* count;    // [B * gamma] chunks of the row whose results are out
  int32_t* part_ids;  // [B * gamma * C * K] chunk top K, ids relative to the chunk
  float* part_logit;  // [B * gamma * C * K]
  float* part_lse;    // [B * gamma * C] chunk LSE
};

// Sweeps work item t (depth-major: position, then sequence, then chunk).
template <typename T>
__device__ __forceinline__ void pipe_worker(const PipeArgs& p, RowLdsT<kPipeWaves>& lds, int t) {
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int per_depth = p.B * p.chunks;
  const int i = t / per_depth;
  const int rem = t - i * per_depth;
  const int b = rem / p.chunks, c = rem - b * p.chunks;
  const int64_t row = static_cast<int64_t>(b) * p.gamma + i;
  const int64_t c0 = static_cast<int64_t>(c) * p.chunk_len;
  const int64_t len = p.V - c0 < p.chunk_len ? p.V - c0 : p.chunk_len;
  const T* rp = static_cast<const T*>(p.logits) + b * p.stride_b + i * p.stride_i + c0;
  sweep_row<T, true, kPipeWaves>(lds, rp, len, p.K, row * p.chunks + c,
                                 RowOut{p.part_ids, p.part_logit, nullptr, p.part_lse, true});
  // Wave 0 wrote the chunk's results with agent-scope atomic stores; once they have
  // completed, the row's counter goes up.
  if (w == 0) {
    wait_all_memory();
    if (lane == 0) __hip_atomic_fetch_add(&p.count[row], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Spins until *f reaches n; false if the wait ran out of time.
__device__ __forceinline__ bool wait_count(const uint32_t* f, uint32_t n, uint64_t t0) {
  for (;;) {
    if (__builtin_amdgcn_readfirstlane(load_agent32(f)) >= n) return true;
    if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) return false;
    __builtin_amdgcn_s_sleep(2);
  }
}

struct SearcherLayout {
  FastLayout fast;
  PipeSearchLayout pipe;
  uint32_t clogit, rready, mstage, total;
};

__host__ __device__ inline SearcherLayout searcher_layout(int gamma, int K, int W) {
  SearcherLayout L{};
  L.fast = fast_layout(gamma, K, W);
  uint32_t q = L.fast.total;
  L.clogit = q;
  q += static_cast<uint32_t>((gamma * K * sizeof(float) + 15) & ~static_cast<size_t>(15));
  L.rready = q;
  q += static_cast<uint32_t>((gamma * sizeof(uint32_t) + 15) & ~static_cast<size_t>(15));
  L.mstage = q;  // one 64-entry order-value stage per wave
  q += static_cast<uint32_t>(kPipeWaves * kWave * sizeof(uint64_t));
  L.pipe = pipe_search_layout(q, gamma);
  L.total = L.pipe.total;
  return L;
}

// Merges the C chunk results of row (b, i) into the row's LSE and sorted top K: lane
// e < C K holds entry e % K of chunk e / K, ranked among all of them by order value (key
// desc, id asc).  Writes the caller's outputs and the candidates into LDS.
template <typename T, int KT>
__device__ __forceinline__ void merge_chunks(const PipeArgs& p, int64_t row, int i, uint64_t* stage, int32_t* cids,
                                             float* clogit, int lane) {
  const int C = p.chunks;
  uint64_t mine = 0;
  int32_t id = 0;
  float v = 0.f;
  if (lane < C * KT) {
    const int c = lane / KT, e = lane - c * KT;
    const int64_t c0 = static_cast<int64_t>(c) * p.chunk_len;
    const int64_t len = p.V - c0 < p.chunk_len ? p.V - c0 : p.chunk_len;
    if (e < len) {
      const int64_t o = (row * C + c) * KT + e;
      id = static_cast<int32_t>(load_agent32(reinterpret_cast<const uint32_t*>(p.part_ids) + o) + c0);
      v = __uint_as_float(load_agent32(reinterpret_cast<const uint32_t*>(p.part_logit) + o));
      mine = cand_order(Traits<T>::key_value(v), static_cast<uint32_t>(id));
    }
  }
  float l = neg_inf();
  if (lane < C) l = __uint_as_float(load_agent32(reinterpret_cast<const uint32_t*>(p.part_lse) + row * C + lane));
  stage[lane] = mine;
  __builtin_amdgcn_wave_barrier();
  const int r = mine != 0 ? count_above(stage, C * KT, mine) : kWave;
  __builtin_amdgcn_wave_barrier();
  // LSE over the chunks, summed in chunk order.
  float m = neg_inf();
  for (int c = 0; c < C; ++c) m = fmaxf(m, __shfl(l, c));
  float e = 0.f;
  for (int c = 0; c < C; ++c) {
    const float lc = __shfl(l, c);
    if (lc != neg_inf()) e += fast_exp2((lc - m) * kLog2e);
  }
  const float lse = (m == neg_inf()) ? neg_inf() : m + fast_log2(e) * kLn2;
  if (r < KT) {
    const int64_t o = row * KT + r;
    cids[i * KT + r] = id;
    clogit[i * KT + r] = v;
    p.cand_ids[o] = id;
    p.cand_logit[o] = v;
    if (p.cand_logprob) p.cand_logprob[o] = v - lse;
  }
  if (lane == 0 && p.lse) p.lse[row] = lse;
}

// A helper wave's positions, w - 1, w - 1 + (nw - 2), ...: it waits for the position's
// chunks, merges them, computes the slab once the predecessor position's candidates are
// in, and publishes it to the search wave.
template <typename T, int KT>
__device__ __forceinline__ void helper_slabs(const PipeArgs& p, const TreeArgs& a, const SelectorArgs& s,
                                             const FastSmem& sm, unsigned char* smem, const SearcherLayout& L, int w,
                                             int nw, int lane) {
  const int b = static_cast<int>(blockIdx.x);
  const int gamma = a.gamma;
  float* clogit = reinterpret_cast<float*>(smem + L.clogit);
  uint32_t* rready = reinterpret_cast<uint32_t*>(smem + L.rready);
  uint64_t* stage = reinterpret_cast<uint64_t*>(smem + L.mstage) + w * kWave;
  const int helpers = nw - 2;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  for (int i = w - 1; i < gamma; i += helpers) {
    const int64_t bi = static_cast<int64_t>(b) * gamma + i;
    if (!wait_count(&p.count[bi], static_cast<uint32_t>(p.chunks), t0) && lane == 0) {
      store_agent32(p.err, 1u);
      __hip_atomic_store(sm.fail, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    merge_chunks<T, KT>(p, bi, i, stage, sm.cids, clogit, lane);
    if (lane == 0) store_agent32(&p.count[bi], 0u);  // read: ready for the next call
    publish_slab(rready, i);
    if (i > 0) wait_flag(&rready[i - 1], sm.fail, t0);
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

// One sequence's merges, selector slabs and tree search.  Wave 0 runs the depth-wise
// expansion, the last wave ranks each frontier and stores it, and the waves between take
// the positions round-robin (helper_slabs).  Then all waves prune, emit and build the mask
// together.
template <typename T, int KT, int R>
__device__ __forceinline__ void searcher(const PipeArgs& p, const TreeArgs& a, const SelectorArgs& s,
                                         uint64_t magic_w, unsigned char* smem, int w, int nw, int lane) {
  const int b = static_cast<int>(blockIdx.x);
  const int gamma = a.gamma;
  const SearcherLayout L = searcher_layout(gamma, KT, a.W);
  const FastSmem sm = fast_smem(smem, L.fast);
  const PipeSearchSmem ps = pipe_search_smem(smem, L.pipe);
  uint32_t* rready = reinterpret_cast<uint32_t*>(smem + L.rready);
  for (int e = static_cast<int>(threadIdx.x); e < gamma; e += static_cast<int>(blockDim.x)) {
    sm.ready[e] = 0u;
    rready[e] = 0u;
    ps.stage_ready[e] = 0u;
    ps.rank_ready[e] = 0u;
  }
  if (threadIdx.x == 0) *sm.fail = 0u;
  __syncthreads();
  __builtin_amdgcn_s_setprio(3);
  if (w == 0)
    pipe_search_wave<KT, R>(a, sm, ps, lane);
  else if (w == nw - 1)
    pipe_prune_wave<KT>(a, sm, ps, lane);
  else
    helper_slabs<T, KT>(p, a, s, sm, smem, L, w, nw, lane);
  finish_tree_coop<KT>(a, sm, ps, b, w, nw, lane, magic_w);
}

// Workgroups 0..B-1 search; workgroup B + t sweeps work item t.
template <typename T, int KT, int R>
__global__ __launch_bounds__(kPipeWaves* kWave, 4) void draft_pipe_kernel(PipeArgs p, TreeArgs a, SelectorArgs s,
                                                                           uint64_t magic_w) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const int lane = static_cast<int>(threadIdx.x) % kWave;
  const int nw = static_cast<int>(blockDim.x) / kWave;
  if (static_cast<int>(blockIdx.x) < p.B) {
    searcher<T, KT, R>(p, a, s, magic_w, smem_raw, w, nw, lane);
    return;
  }
  pipe_worker<T>(p, *reinterpret_cast<RowLdsT<kPipeWaves>*>(smem_raw), static_cast<int>(blockIdx.x) - p.B);
}

int compute_units() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

// Chunks per row and elements per chunk: at most kPipeMaxChunks chunks with C K <= 64, each a
// whole number of tiles; no chunk is empty.
void pipe_chunks(int64_t V, int K, int dtype, int& C, int64_t& len) {
  const int64_t tile = static_cast<int64_t>(kSubGroups) * kWave * (dtype == 1 ? 8 : 4);
  const int64_t tiles = (V + tile - 1) / tile;
  int c = kPipeMaxChunks;
  while (c > 1 && c * K > kWave) --c;
  if (c > tiles) c = static_cast<int>(tiles);
  len = (tiles + c - 1) / c * tile;
  C = static_cast<int>((V + len - 1) / len);
}

size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

struct PipeWorkspace {
  size_t count, part_ids, part_logit, part_lse, total;
};

PipeWorkspace pipe_workspace(int B, int gamma, int64_t V, int K, int dtype) {
  int C = 1;
  int64_t len = 0;
  pipe_chunks(V, K, dtype, C, len);
  const size_t rows = static_cast<size_t>(B) * gamma;
  PipeWorkspace w{};
  w.count = kCountBase;
  w.part_ids = w.count + align256(rows * sizeof(uint32_t));
  w.part_logit = w.part_ids + align256(rows * C * K * sizeof(int32_t));
  w.part_lse = w.part_logit + align256(rows * C * K * sizeof(float));
  w.total = w.part_lse + align256(rows * C * sizeof(float));
  return w;
}

// Largest workspace of the one-launch shapes: B <= kMaxStepSequences, gamma <= 64 and
// K <= 16 with at most kPipeMaxChunks chunks per row (V and the dtype do not change it).
constexpr size_t kStaticRows = static_cast<size_t>(kMaxStepSequences) * 64;
constexpr size_t kStaticScratchBytes = kCountBase + ((kStaticRows * 4 + 255) & ~size_t(255)) +
                                       2 * ((kStaticRows * kPipeMaxChunks * 16 * 4 + 255) & ~size_t(255)) +
                                       ((kStaticRows * kPipeMaxChunks * 4 + 255) & ~size_t(255));

// The allocation-free variant's workspace: one array per device, held until the process
// ends.  Host code never passes this name to a kernel (on the host it is only a stand-in
// for the symbol); it uses the device address hipGetSymbolAddress returns for the device.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Zero-fills n 32-bit words (a fill kernel rather than a memset, so graph capture records
// a kernel node).
__global__ void zero_words_kernel(uint32_t* __restrict__ p, int n) {
  const int i = static_cast<int>(blockIdx.x * blockDim.x + threadIdx.x);
  if (i < n) p[i] = 0u;
}

}  // namespace

// ---- host side ------------------------------------------------------------------------------
size_t step_static_scratch_bytes() { return kStaticScratchBytes; }

hipError_t step_static_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t clear_step_flags(void* workspace, int B, int gamma, hipStream_t stream) {
  // The error word (and the rest of the first 256 bytes) and one counter per row.
  const int words = static_cast<int>(kCountBase / 4) + B * gamma;
  hipLaunchKernelGGL(zero_words_kernel, dim3(static_cast<unsigned>((words + 255) / 256)), dim3(256), 0, stream,
                     static_cast<uint32_t*>(workspace), words);
  return hipGetLastError();
}

size_t step_workspace_bytes(int B, int gamma, int64_t V, int K, int dtype) {
  return pipe_workspace(B, gamma, V, K, dtype).total;
}

bool draft_step_fused(int dtype, bool aligned, int B, int gamma, int64_t V, int K, int feat_dtype, int W) {
  if (!aligned || feat_dtype != 1 || B > kMaxStepSequences) return false;
  if (!draft_tree_fused(feat_dtype, gamma, K, W)) return false;
  (void)dtype;
  (void)V;
  const int cus = compute_units();
  return cus > 0 && B < cus;
}

bool draft_step_k64(int feat_dtype, int B, int gamma, int K, int W) {
  if (B > kMaxStepSequences || !draft_tree_k64_fused(feat_dtype, gamma, K, W)) return false;
  const int cus = compute_units();
  return cus > 0 && B < cus;
}

size_t step_k64_workspace_bytes(int B, int gamma) {
  return kCountBase + align256(static_cast<size_t>(B) * gamma * sizeof(uint32_t));
}

hipError_t launch_draft_step_k64(const SelectorArgs& s, const TreeArgs& a, void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  TreeArgs ta = a;
  ta.err = reinterpret_cast<uint32_t*>(ws);  // a search that ran out of time sets the error word
  return launch_draft_tree_k64(s, ta, reinterpret_cast<uint32_t*>(ws + kCountBase), stream);
}

hipError_t launch_draft_step(const void* logits, int dtype, int B, int gamma, int64_t V, int64_t stride_b,
                             int64_t stride_i, int K, int32_t* cand_ids, float* cand_logit, float* cand_logprob,
                             float* lse, const SelectorArgs& s, const TreeArgs& a, void* workspace,
                             hipStream_t stream) {
  PipeArgs p{};
  p.logits = logits;
  p.V = V;
  p.stride_b = stride_b;
  p.stride_i = stride_i;
  p.B = B;
  p.gamma = gamma;
  p.K = K;
  pipe_chunks(V, K, dtype, p.chunks, p.chunk_len);
  p.cand_ids = cand_ids;
  p.cand_logit = cand_logit;
  p.cand_logprob = cand_logprob;
  p.lse = lse;
  const PipeWorkspace pw = pipe_workspace(B, gamma, V, K, dtype);
  char* ws = static_cast<char*>(workspace);
  p.err = reinterpret_cast<uint32_t*>(ws);
  p.count = reinterpret_cast<uint32_t*>(ws + pw.count);
  p.part_ids = reinterpret_cast<int32_t*>(ws + pw.part_ids);
  p.part_logit = reinterpret_cast<float*>(ws + pw.part_logit);
  p.part_lse = reinterpret_cast<float*>(ws + pw.part_lse);
  TreeArgs ta = a;
  ta.err = p.err;  // a search that ran out of time also sets the workspace's error word

  const uint64_t magic_w = (0x100000000ull + a.W - 1) / a.W;
  const size_t row_smem = sizeof(RowLdsT<kPipeWaves>);
  const size_t search_smem = searcher_layout(gamma, K, a.W).total;
  const size_t smem = row_smem > search_smem ? row_smem : search_smem;
  const dim3 grid(static_cast<unsigned>(B + B * gamma * p.chunks));
  const dim3 block(kPipeWaves * kWave);
  const int wk = a.W * K;
#define UBT_PIPE_LAUNCH(TT, KK, RR)                                                                         \
  do {                                                                                                      \
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&draft_pipe_kernel<TT, KK, RR>),               \
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));          \
    hipLaunchKernelGGL((draft_pipe_kernel<TT, KK, RR>), grid, block, smem, stream, p, ta, s, magic_w);      \
  } while (0)
#define UBT_PIPE_ROWS(TT, KK)       \
  do {                              \
    if (wk <= 64)                   \
      UBT_PIPE_LAUNCH(TT, KK, 1);   \
    else if (wk <= 128)             \
      UBT_PIPE_LAUNCH(TT, KK, 2);   \
    else if (wk <= 256)             \
      UBT_PIPE_LAUNCH(TT, KK, 4);   \
    else if (wk <= 384)             \
      UBT_PIPE_LAUNCH(TT, KK, 6);   \
    else                            \
      UBT_PIPE_LAUNCH(TT, KK, 8);   \
  } while (0)
#define UBT_PIPE_K(TT)         \
  do {                         \
    if (K == 4)                \
      UBT_PIPE_ROWS(TT, 4);    \
    else if (K == 8)           \
      UBT_PIPE_ROWS(TT, 8);    \
    else                       \
      UBT_PIPE_ROWS(TT, 16);   \
  } while (0)
  if (dtype == 1)
    UBT_PIPE_K(uint16_t);
  else
    UBT_PIPE_K(float);
#undef UBT_PIPE_K
#undef UBT_PIPE_ROWS
#undef UBT_PIPE_LAUNCH
  return hipGetLastError();
}

}  // namespace ubt
