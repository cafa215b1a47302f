// TEST INFRASTRUCTURE -- plain, slow fp64 CPU oracle for the UBTree draft-tree
// construction step (arXiv 2609.39972).  Only the test-suite, the smoke check and the
// CPU-baseline leg of the benchmark load this library.  The HIP product library never
// links, loads or calls it, and the two share no code: not a header, helper, table or
// constant.
//
// Each entry point follows one passage of the paper, in the paper's order and notation:
//
//   ubt_oracle_topk        Method / Unigram Proposer (Eq. ubtree-unigram) and
//                          "Candidate Sets": C_i = the top-K tokens of q_i = softmax(u_i).
//   ubt_oracle_bigram      Background (Eq. dflash2-selector): delta_i(a,b) =
//                          (P(h_i) (.) phi(a))^T psi(b); Method / Depth Calibration
//                          (Eq. ubtree-depth): s_i = alpha_i u_i(b) + lambda_i delta_i(a,b);
//                          Method / Parallel Computation (Eq. ubtree-edge-matrix): all pairs
//                          of C_{i-1} x C_i with C_0 = {x_0}; Appendix A / Path Scores
//                          (Eq. ubtree-path): log q_i^bi(b|a) = s_i(a,b) - log sum_v exp s_i(a,v).
//   ubt_oracle_build_tree  Appendix A: Depth Bonus (Eq. ubtree-depth-bonus), Depth-Wise
//                          Expansion (Eq. ubtree-frontier), Global Pruning (Eq. ubtree-pruning)
//                          and Algorithm 1 (construction from precomputed scores).
//   ubt_oracle_tree_mask   Appendix A / Verification via Tree-attention: every node attends
//                          to itself and to its ancestors.
//   ubt_oracle_edge_scores, ubt_oracle_best_first
//                          the unigram-plus-bigram scoring: each edge scores its
//                          successor's unigram log-probability (Eq. ubtree-unigram) plus its
//                          raw selector score (Eq. dflash2-selector), weighted as in Eq.
//                          ubtree-depth; paths are ranked by the cumulative sum and grown
//                          best-first (Background, "Tree Drafting": best-first search over
//                          accumulated scores).  These sums are not monotone along a path,
//                          so the prefix closure that Appendix A / Global Pruning gets from
//                          normalisation is enforced by the search itself: a node becomes
//                          eligible only once its parent is in the tree.
//
// Readings where the paper is silent (each is listed with its reason in the design notes):
//   * ties in C_i go to the lower token id; values compare as real numbers (-0 == +0);
//   * ties inside Top_W / Top_B: "prefer ancestors" is realised by the total order
//       within a depth: score desc, then the parent's position in F_{d-1}, then the
//       candidate rank c; across depths: score desc, then depth asc, then that order;
//   * the non-root budget B excludes the root, which is emitted at slot 0;
//   * logarithms are natural; every sum runs in fp64 in index order.
//
// Status codes: 0 ok, 1 bad arguments, 2 a selected node's parent was not selected
// (the prefix-closure lemma of Appendix A says this cannot happen).

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <numeric>
#include <thread>
#include <vector>

namespace {

const double kNegInf = -std::numeric_limits<double>::infinity();

// Exact decode of one stored element: dtype 0 = IEEE binary32, 1 = bfloat16 (the upper
// 16 bits of a binary32).
double load_value(const void* base, int dtype, int64_t i) {
  if (dtype == 0) return static_cast<double>(static_cast<const float*>(base)[i]);
  uint32_t bits = static_cast<uint32_t>(static_cast<const uint16_t*>(base)[i]) << 16;
  float f;
  std::memcpy(&f, &bits, sizeof f);
  return static_cast<double>(f);
}

// Runs body(i) for i in [0, n) on up to n_threads threads (static round-robin split).
template <class Body>
void parallel_for(int64_t n, int n_threads, Body body) {
  const int64_t T = std::max<int64_t>(1, std::min<int64_t>(n_threads, n));
  if (T == 1) {
    for (int64_t i = 0; i < n; ++i) body(i);
    return;
  }
  std::vector<std::thread> pool;
  for (int64_t t = 0; t < T; ++t)
    pool.emplace_back([=] {
      for (int64_t i = t; i < n; i += T) body(i);
    });
  for (auto& th : pool) th.join();
}

// log sum_j exp(x_j), shifted by the maximum.
double log_sum_exp(const std::vector<double>& x) {
  double m = kNegInf;
  for (double v : x) m = std::max(m, v);
  if (m == kNegInf) return kNegInf;
  double s = 0.0;
  for (double v : x) s += std::exp(v - m);
  return m + std::log(s);
}

}  // namespace

extern "C" {

int ubt_oracle_version(void) { return 1; }

// Candidate selection and softmax statistics for `rows` rows of V logits stored
// contiguously.  Per row: cand_ids = the K largest logits, ordered by (logit desc, id asc);
// cand_logit = those logits; lse = log sum_v exp(u_v); cand_logprob = cand_logit - lse,
// i.e. log q_i of each candidate.  Ranking u ranks q_i, because softmax is increasing.
int ubt_oracle_topk(const void* logits, int dtype, int64_t rows, int64_t V, int K,
                    int32_t* cand_ids, double* cand_logit, double* cand_logprob, double* lse,
                    int n_threads) {
  if (!logits || !cand_ids || !cand_logit || !cand_logprob || !lse) return 1;
  if ((dtype != 0 && dtype != 1) || rows < 0 || V < 1 || K < 1 || K > V) return 1;
  parallel_for(rows, n_threads, [&](int64_t row) {
    std::vector<double> u(static_cast<size_t>(V));
    for (int64_t v = 0; v < V; ++v) u[v] = load_value(logits, dtype, row * V + v);

    std::vector<int32_t> order(static_cast<size_t>(V));
    std::iota(order.begin(), order.end(), 0);
    std::partial_sort(order.begin(), order.begin() + K, order.end(), [&](int32_t a, int32_t b) {
      return u[a] > u[b] || (u[a] == u[b] && a < b);
    });

    const double l = log_sum_exp(u);
    lse[row] = l;
    for (int k = 0; k < K; ++k) {
      const int32_t id = order[k];
      cand_ids[row * K + k] = id;
      cand_logit[row * K + k] = u[id];
      cand_logprob[row * K + k] = u[id] - l;
    }
  });
  return 0;
}

// Selector scores and normalised transition log-probabilities.  Layouts (row-major):
// phi_tab, psi_tab [V, r]; gate [B, gamma, r]; cand_ids, cand_logit [B, gamma, K];
// alpha, lambda [gamma]; delta, logq [B, gamma, K, K] indexed [b][i][a][c], where position
// i = 0..gamma-1 is draft depth i+1, a indexes the predecessor set and c the successor
// candidate rank.  At i = 0 the predecessor set is {anchor[b]} (row a = 0); rows
// a = 1..K-1 of that slab are written as 0.
int ubt_oracle_bigram(const void* phi_tab, const void* psi_tab, const void* gate, int feat_dtype,
                      int64_t V, int r, const int32_t* anchor, const int32_t* cand_ids,
                      const double* cand_logit, const double* alpha, const double* lambda,
                      int B, int gamma, int K, double* delta, double* logq, int n_threads) {
  if (!phi_tab || !psi_tab || !gate || !anchor || !cand_ids || !cand_logit || !alpha ||
      !lambda || !delta || !logq)
    return 1;
  if ((feat_dtype != 0 && feat_dtype != 1) || V < 1 || r < 1 || B < 0 || gamma < 1 || K < 1)
    return 1;
  parallel_for(static_cast<int64_t>(B) * gamma, n_threads, [&](int64_t bi) {
    const int64_t b = bi / gamma;
    const int i = static_cast<int>(bi % gamma);
    const int n_pred = (i == 0) ? 1 : K;
    double* dslab = delta + bi * K * K;
    double* qslab = logq + bi * K * K;
    std::fill(dslab, dslab + static_cast<int64_t>(K) * K, 0.0);
    std::fill(qslab, qslab + static_cast<int64_t>(K) * K, 0.0);
    for (int a = 0; a < n_pred; ++a) {
      const int64_t pred = (i == 0) ? anchor[b] : cand_ids[(bi - 1) * K + a];
      std::vector<double> s(static_cast<size_t>(K));
      for (int c = 0; c < K; ++c) {
        const int64_t succ = cand_ids[bi * K + c];
        // delta_i(a, b) = sum_k P(h_i)_k * phi_k(a) * psi_k(b)
        double d = 0.0;
        for (int k = 0; k < r; ++k)
          d += load_value(gate, feat_dtype, bi * r + k) * load_value(phi_tab, feat_dtype, pred * r + k) *
               load_value(psi_tab, feat_dtype, succ * r + k);
        dslab[a * K + c] = d;
        // s_i(a, b) = alpha_i u_i(b) + lambda_i delta_i(a, b)
        s[c] = alpha[i] * cand_logit[bi * K + c] + lambda[i] * d;
      }
      // log q_i^bi(b | a): normalise over the successor candidates C_i.
      const double norm = log_sum_exp(s);
      for (int c = 0; c < K; ++c) qslab[a * K + c] = s[c] - norm;
    }
  });
  return 0;
}

// Algorithm 1 for B independent sequences.  Inputs: anchor [B], cand_ids [B, gamma, K],
// logq [B, gamma, K, K] as written by ubt_oracle_bigram, search width W, non-root budget
// `budget`, depth bonus zeta <= 0.  Outputs, N = budget + 1 slots per sequence, root at
// slot 0 and the selected nodes after it in selection order:
//   n_nodes [B]; token, parent, depth, cand_rank [B, N] (int32, -1 in unused slots);
//   score [B, N] (fp64, -inf in unused slots); mask [B, N, ceil(N/32)] (uint32, bit m%32
//   of word m/32 set iff slot m is slot n or one of its ancestors).
// Optional supertree dump (any pointer may be null): f_count [B, gamma] = |F_d|;
// f_parent, f_cand [B, gamma, W] = parent position in F_{d-1} and candidate rank c of the
// j-th member of F_d; f_score [B, gamma, W]; unused entries -1 / -inf.
int ubt_oracle_build_tree(const int32_t* anchor, const int32_t* cand_ids, const double* logq,
                          int B, int gamma, int K, int W, int budget, double zeta,
                          int32_t* n_nodes, int32_t* token, int32_t* parent, int32_t* depth,
                          int32_t* cand_rank, double* score, uint32_t* mask, int32_t* f_count,
                          int32_t* f_parent, int32_t* f_cand, double* f_score, int n_threads) {
  if (!anchor || !cand_ids || !logq || !n_nodes || !token || !parent || !depth || !cand_rank ||
      !score || !mask)
    return 1;
  if (B < 0 || gamma < 1 || K < 1 || W < 1 || budget < 1 || !(zeta <= 0.0)) return 1;
  const int N = budget + 1;
  const int words = (N + 31) / 32;
  std::vector<int> status(static_cast<size_t>(B), 0);

  parallel_for(B, n_threads, [&](int64_t b) {
    struct Node {
      double score;  // l_zeta of the node's prefix
      int parent;    // position of the parent in F_{d-1} (-1 for the root)
      int c;         // candidate rank within C_d (-1 for the root)
    };
    // F[0] = {epsilon} with l_zeta(epsilon) = 0.
    std::vector<std::vector<Node>> F(static_cast<size_t>(gamma) + 1);
    F[0].push_back({0.0, -1, -1});

    for (int d = 1; d <= gamma; ++d) {
      // E_d: every retained prefix of depth d-1 extended by every candidate of C_d,
      // listed parent-major (parents in F_{d-1} order), candidate-minor.
      std::vector<Node> E;
      for (int p = 0; p < static_cast<int>(F[d - 1].size()); ++p) {
        // The predecessor token of the extension: the anchor x_0 at depth 1 (row 0 of
        // the slab), otherwise the parent's own candidate.
        const int row = (d == 1) ? 0 : F[d - 1][p].c;
        const double* q = logq + ((b * gamma + (d - 1)) * static_cast<int64_t>(K) + row) * K;
        for (int c = 0; c < K; ++c) E.push_back({F[d - 1][p].score + q[c] + zeta, p, c});
      }
      // F_d = Top_W(E_d; l_zeta): the W best extensions over all parents.  A stable
      // sort keeps the E_d order (parent order, then c) among equal scores.
      std::stable_sort(E.begin(), E.end(), [](const Node& x, const Node& y) { return x.score > y.score; });
      E.resize(std::min<size_t>(E.size(), static_cast<size_t>(W)));
      F[d] = E;
    }

    // S = union of F_d; T = {epsilon} + Top_B(S; l_zeta).  S is listed depth by depth in
    // F_d order, so a stable sort by score keeps (depth asc, F_d order) among ties.
    struct Ref {
      double score;
      int d, j;
    };
    std::vector<Ref> S;
    for (int d = 1; d <= gamma; ++d)
      for (int j = 0; j < static_cast<int>(F[d].size()); ++j) S.push_back({F[d][j].score, d, j});
    std::stable_sort(S.begin(), S.end(), [](const Ref& x, const Ref& y) { return x.score > y.score; });
    const int n_sel = std::min<int>(static_cast<int>(S.size()), budget);

    int32_t* tok = token + b * N;
    int32_t* par = parent + b * N;
    int32_t* dep = depth + b * N;
    int32_t* cr = cand_rank + b * N;
    double* sc = score + b * N;
    for (int n = 0; n < N; ++n) {
      tok[n] = par[n] = dep[n] = cr[n] = -1;
      sc[n] = kNegInf;
    }
    // Root: the anchor token, depth 0, score 0.
    tok[0] = anchor[b];
    dep[0] = 0;
    sc[0] = 0.0;

    std::vector<std::vector<int>> slot(static_cast<size_t>(gamma) + 1);
    for (int d = 0; d <= gamma; ++d) slot[d].assign(F[d].size(), -1);
    slot[0][0] = 0;
    for (int n = 1; n <= n_sel; ++n) {
      const Ref& x = S[n - 1];
      const Node& node = F[x.d][x.j];
      const int ps = slot[x.d - 1][node.parent];
      if (ps < 0) status[b] = 2;  // parent not selected before its child
      slot[x.d][x.j] = n;
      tok[n] = cand_ids[(b * gamma + (x.d - 1)) * static_cast<int64_t>(K) + node.c];
      par[n] = ps;
      dep[n] = x.d;
      cr[n] = node.c;
      sc[n] = node.score;
    }
    n_nodes[b] = 1 + n_sel;

    // Ancestor mask: walk each node's parent chain up to the root.
    uint32_t* mrow = mask + b * static_cast<int64_t>(N) * words;
    std::fill(mrow, mrow + static_cast<int64_t>(N) * words, 0u);
    for (int n = 0; n <= n_sel; ++n)
      for (int m = n; m >= 0; m = par[m]) mrow[n * words + m / 32] |= 1u << (m % 32);

    if (f_count)
      for (int d = 1; d <= gamma; ++d) f_count[b * gamma + d - 1] = static_cast<int32_t>(F[d].size());
    for (int d = 1; d <= gamma; ++d)
      for (int j = 0; j < W; ++j) {
        const int64_t o = (b * gamma + (d - 1)) * static_cast<int64_t>(W) + j;
        const bool have = j < static_cast<int>(F[d].size());
        if (f_parent) f_parent[o] = have ? F[d][j].parent : -1;
        if (f_cand) f_cand[o] = have ? F[d][j].c : -1;
        if (f_score) f_score[o] = have ? F[d][j].score : kNegInf;
      }
  });
  for (int s : status)
    if (s) return s;
  return 0;
}

// Edge scores of the unigram-plus-bigram scoring.  Inputs as written by ubt_oracle_topk
// (cand_logprob = log q_i of each candidate, i.e. u - LSE) and ubt_oracle_bigram (delta,
// [B, gamma, K, K] indexed [b][i][a][c]); alpha, lambda [gamma].  Output edge [B, gamma,
// K, K], same indexing:
//   e_i(a, c) = alpha_i * log q_i(C_i[c]) + lambda_i * delta_i(a, c)
// with no normalisation over the successors.  At i = 0 only row a = 0 (the anchor) is a
// predecessor; rows 1..K-1 of that slab are written as 0.
int ubt_oracle_edge_scores(const double* cand_logprob, const double* delta, const double* alpha,
                           const double* lambda, int B, int gamma, int K, double* edge) {
  if (!cand_logprob || !delta || !alpha || !lambda || !edge || B < 0 || gamma < 1 || K < 1) return 1;
  for (int64_t b = 0; b < B; ++b)
    for (int i = 0; i < gamma; ++i) {
      const int64_t bi = b * gamma + i;
      const int n_pred = (i == 0) ? 1 : K;
      for (int a = 0; a < K; ++a)
        for (int c = 0; c < K; ++c) {
          const int64_t o = (bi * K + a) * K + c;
          edge[o] = (a < n_pred) ? alpha[i] * cand_logprob[bi * K + c] + lambda[i] * delta[o] : 0.0;
        }
    }
  return 0;
}

// Best-first tree over the candidate lattice for B independent sequences.  Inputs:
// anchor [B], cand_ids [B, gamma, K], edge [B, gamma, K, K] (any real values; e.g. from
// ubt_oracle_edge_scores), non-root budget, depth bonus zeta <= 0.
// The path score is l(y_{1:d}) = sum_{i<=d} e_i(y_{i-1}, y_i) + zeta * d, with y_0 the
// anchor (row 0 of the first slab).  Starting from the root, the tree grows one node at a
// time: among the children of tree nodes that are not yet in the tree (the frontier), the
// best one is added, under the order
//   score desc, then depth asc, then the parent's slot asc, then candidate rank asc,
// until `budget` nodes are in or the frontier is empty.  Slots are assigned in that
// addition order (root = 0), so every parent precedes its children.  Outputs as for
// ubt_oracle_build_tree (no supertree).
int ubt_oracle_best_first(const int32_t* anchor, const int32_t* cand_ids, const double* edge,
                          int B, int gamma, int K, int budget, double zeta,
                          int32_t* n_nodes, int32_t* token, int32_t* parent, int32_t* depth,
                          int32_t* cand_rank, double* score, uint32_t* mask, int n_threads) {
  if (!anchor || !cand_ids || !edge || !n_nodes || !token || !parent || !depth || !cand_rank ||
      !score || !mask)
    return 1;
  if (B < 0 || gamma < 1 || K < 1 || budget < 1 || !(zeta <= 0.0)) return 1;
  const int N = budget + 1;
  const int words = (N + 31) / 32;

  parallel_for(B, n_threads, [&](int64_t b) {
    struct Cand {
      double score;  // l of the candidate node's prefix
      int depth;     // its depth d >= 1
      int pslot;     // slot of its parent in the tree
      int c;         // its candidate rank in C_d
    };
    auto before = [](const Cand& x, const Cand& y) {
      if (x.score != y.score) return x.score > y.score;
      if (x.depth != y.depth) return x.depth < y.depth;
      if (x.pslot != y.pslot) return x.pslot < y.pslot;
      return x.c < y.c;
    };
    int32_t* tok = token + b * N;
    int32_t* par = parent + b * N;
    int32_t* dep = depth + b * N;
    int32_t* cr = cand_rank + b * N;
    double* sc = score + b * N;
    for (int n = 0; n < N; ++n) {
      tok[n] = par[n] = dep[n] = cr[n] = -1;
      sc[n] = kNegInf;
    }
    tok[0] = anchor[b];
    dep[0] = 0;
    sc[0] = 0.0;

    // The children of a tree node at slot `slot` (depth d, candidate rank c; the root has
    // d = 0 and predecessor row 0): the K candidates of position d + 1.
    std::vector<Cand> frontier;
    auto push_children = [&](int slot, int d, int c, double s) {
      if (d >= gamma) return;
      const int row = (d == 0) ? 0 : c;
      const double* e = edge + ((b * gamma + d) * static_cast<int64_t>(K) + row) * K;
      for (int k = 0; k < K; ++k) frontier.push_back({s + e[k] + zeta, d + 1, slot, k});
    };
    push_children(0, 0, -1, 0.0);
    int n = 1;
    while (n <= budget && !frontier.empty()) {
      size_t best = 0;
      for (size_t j = 1; j < frontier.size(); ++j)
        if (before(frontier[j], frontier[best])) best = j;
      const Cand x = frontier[best];
      frontier.erase(frontier.begin() + static_cast<std::ptrdiff_t>(best));
      tok[n] = cand_ids[(b * gamma + (x.depth - 1)) * static_cast<int64_t>(K) + x.c];
      par[n] = x.pslot;
      dep[n] = x.depth;
      cr[n] = x.c;
      sc[n] = x.score;
      push_children(n, x.depth, x.c, x.score);
      ++n;
    }
    n_nodes[b] = n;

    uint32_t* mrow = mask + b * static_cast<int64_t>(N) * words;
    std::fill(mrow, mrow + static_cast<int64_t>(N) * words, 0u);
    for (int m0 = 0; m0 < n; ++m0)
      for (int m = m0; m >= 0; m = par[m]) mrow[m0 * words + m / 32] |= 1u << (m % 32);
  });
  return 0;
}

// Ancestor mask from parent pointers: parent [B, N] with parent[0] = -1 and
// parent[n] < n for 1 <= n < n_nodes[b]; mask [B, N, ceil(N/32)], rows >= n_nodes zero.
int ubt_oracle_tree_mask(const int32_t* parent, const int32_t* n_nodes, int B, int N, uint32_t* mask) {
  if (!parent || !n_nodes || !mask || B < 0 || N < 1) return 1;
  const int words = (N + 31) / 32;
  for (int64_t b = 0; b < B; ++b) {
    uint32_t* mrow = mask + b * static_cast<int64_t>(N) * words;
    std::fill(mrow, mrow + static_cast<int64_t>(N) * words, 0u);
    const int32_t* par = parent + b * N;
    const int lim = std::min(n_nodes[b], N);
    for (int n = 0; n < lim; ++n) {
      int m = n;
      while (true) {
        mrow[n * words + m / 32] |= 1u << (m % 32);
        if (m == 0) break;  // reached the root
        const int p = par[m];
        if (p < 0 || p >= m) return 1;  // parents must precede their children
        m = p;
      }
    }
  }
  return 0;
}

}  // extern "C"
