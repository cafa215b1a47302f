// UBTree's renormalised-KL training objective and its gradients.
//
// Method / Tree-native Training, Eq. (ubtree-training-distributions): on the proposer's
// top-K support C_i, p~ = softmax(z_i / T) of the target logits (T -> 0+: uniform over
// their maximisers) and q~ = softmax(s_i(y*_{i-1}, .)) of the selector logits given the
// ground-truth predecessor; Eq. (ubtree-training-loss): loss = KL(p~ || q~) - beta log
// q_i(y*_i), the second term on the proposer's full-vocabulary softmax.  The selector
// logit is s = alpha_i u_i(b) + lambda_i delta_i(a, b) (Depth Calibration, Eq.
// (ubtree-depth)) with delta_i(a, b) = (P(h_i) * phi(a)) . psi(b) (Background, Eq.
// (dflash2-selector)).  Gradients:
//   d loss / d s(b)   = q~(b) - p~(b)
//   d loss / d u_i(v) = beta (softmax(u_i)(v) - [v = y*_i]) + alpha_i [v in C_i] (q~ - p~)(v)
//
// Two launches.  The dense one streams every logit row once and writes
// beta * exp(u - LSE) (HBM-bound: read the row, write fp32).  The per-position one (one
// wave per row) forms delta for the K candidates, the two distributions, the loss terms
// and d loss / d s, then adds the K + 1 sparse terms of the logit gradient to what the
// dense launch wrote (stream order makes those writes visible).
#include "ubt_device.h"
#include "ubt_launch.h"

namespace ubt {
namespace {

typedef uint32_t w4u __attribute__((ext_vector_type(4)));
typedef float w4f __attribute__((ext_vector_type(4)));

constexpr int kDenseThreads = 256;
constexpr int kDenseUnroll = 4;  // 8-element groups per thread per pass, in flight together

template <typename T>
__device__ __forceinline__ float logit_at(const T* p, int64_t i);
template <>
__device__ __forceinline__ float logit_at<float>(const float* p, int64_t i) {
  return p[i];
}
template <>
__device__ __forceinline__ float logit_at<uint16_t>(const uint16_t* p, int64_t i) {
  return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}

__device__ __forceinline__ bool valid_token(int32_t y, int64_t V) { return y >= 0 && y < V; }

// grad[row][v] = beta * exp(u[row][v] - lse[row]) for valid rows, 0 for invalid ones.
// Grid: (B * gamma rows, chunks of kDenseThreads * 8 * kDenseUnroll elements).
template <typename T, bool kVec>
__global__ __launch_bounds__(kDenseThreads) void kl_dense_kernel(const T* __restrict__ logits, int gamma, int64_t V,
                                                                 int64_t stride_b, int64_t stride_i,
                                                                 const float* __restrict__ lse,
                                                                 const int32_t* __restrict__ y_star, float beta,
                                                                 float* __restrict__ grad) {
  const int64_t row = blockIdx.x;
  const int64_t b = row / gamma, i = row - b * gamma;
  const T* u = logits + b * stride_b + i * stride_i;
  float* g = grad + row * V;
  const bool valid = valid_token(y_star[row], V);
  const float shift = valid ? lse[row] * kLog2e : 0.f;
  constexpr int64_t kChunk = static_cast<int64_t>(kDenseThreads) * 8 * kDenseUnroll;
  const int64_t c0 = static_cast<int64_t>(blockIdx.y) * kChunk;
  if (kVec) {
    // Whole 8-element groups (V % 8 == 0 and 16-byte aligned rows).
    float x[kDenseUnroll][8];
#pragma unroll
    for (int k = 0; k < kDenseUnroll; ++k) {
      const int64_t e = c0 + (static_cast<int64_t>(k) * kDenseThreads + threadIdx.x) * 8;
      if (e < V) {
        if (sizeof(T) == 2) {
          const w4u v = *reinterpret_cast<const w4u*>(u + e);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            x[k][2 * j] = __uint_as_float(v[j] << 16);
            x[k][2 * j + 1] = __uint_as_float(v[j] & 0xFFFF0000u);
          }
        } else {
          const w4f v0 = *reinterpret_cast<const w4f*>(u + e);
          const w4f v1 = *reinterpret_cast<const w4f*>(u + e + 4);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            x[k][j] = v0[j];
            x[k][4 + j] = v1[j];
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kDenseUnroll; ++k) {
      const int64_t e = c0 + (static_cast<int64_t>(k) * kDenseThreads + threadIdx.x) * 8;
      if (e < V) {
        float y[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = valid ? beta * __builtin_amdgcn_exp2f(fmaf(x[k][j], kLog2e, -shift)) : 0.f;
        *reinterpret_cast<w4f*>(g + e) = w4f{y[0], y[1], y[2], y[3]};
        *reinterpret_cast<w4f*>(g + e + 4) = w4f{y[4], y[5], y[6], y[7]};
      }
    }
  } else {
    for (int64_t e = c0 + threadIdx.x; e < V && e < c0 + kChunk; e += kDenseThreads)
      g[e] = valid ? beta * __builtin_amdgcn_exp2f(fmaf(logit_at<T>(u, e), kLog2e, -shift)) : 0.f;
  }
}

// Features k..k+7 of a row (16-byte aligned: rows hold a multiple of 16 features).
template <typename F>
__device__ __forceinline__ void feat8(const F* p, int k, float (&x)[8]);
template <>
__device__ __forceinline__ void feat8<float>(const float* p, int k, float (&x)[8]) {
  const w4f a = *reinterpret_cast<const w4f*>(p + k), b = *reinterpret_cast<const w4f*>(p + k + 4);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    x[j] = a[j];
    x[4 + j] = b[j];
  }
}
template <>
__device__ __forceinline__ void feat8<uint16_t>(const uint16_t* p, int k, float (&x)[8]) {
  const w4u v = *reinterpret_cast<const w4u*>(p + k);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    x[2 * j] = __uint_as_float(v[j] << 16);
    x[2 * j + 1] = __uint_as_float(v[j] & 0xFFFF0000u);
  }
}

struct LossArgs {
  const void* logits;
  const void* target;
  int gamma, K, r;
  int64_t V, stride_b, stride_i, t_stride_b, t_stride_i;
  const float* lse;
  const int32_t* cand_ids;
  const float* cand_logit;
  const int32_t* y_star;
  const int32_t* anchor;
  const void* phi;
  const void* psi;
  const void* gate;
  Scales sc;
  float inv_T;  // 1 / T, or 0 for T = 0
  float beta;
  float* loss;
  float* kl;
  float* ce;
  float* grad_s;
  float* grad;
};

// One wave per (sequence, position); lane j < K holds candidate j.
template <typename T, typename F>
__global__ __launch_bounds__(kWave) void kl_position_kernel(LossArgs p) {
  const int64_t row = blockIdx.x;
  const int b = static_cast<int>(row / p.gamma), i = static_cast<int>(row % p.gamma);
  const int lane = static_cast<int>(threadIdx.x);
  const int K = p.K;
  const bool on = lane < K;
  const int32_t y = p.y_star[row];
  if (!valid_token(y, p.V)) {
    if (lane == 0) {
      p.loss[row] = 0.f;
      if (p.kl) p.kl[row] = 0.f;
      if (p.ce) p.ce[row] = 0.f;
    }
    if (on && p.grad_s) p.grad_s[row * K + lane] = 0.f;
    return;
  }
  const int32_t a = i == 0 ? p.anchor[b] : p.y_star[row - 1];
  const bool has_pred = valid_token(a, p.V);
  const int32_t cid = on ? p.cand_ids[row * K + lane] : 0;
  const bool cin = on && valid_token(cid, p.V);
  const int64_t c = cin ? cid : 0;

  // delta(a, c) = sum_k gate_k phi_k(a) psi_k(c): the products are exact in fp32 for
  // bf16 features; the sum runs in k order.
  float delta = 0.f;
  if (has_pred) {
    const F* g = static_cast<const F*>(p.gate) + row * p.r;
    const F* ph = static_cast<const F*>(p.phi) + static_cast<int64_t>(a) * p.r;
    const F* ps = static_cast<const F*>(p.psi) + c * p.r;
    for (int k = 0; k < p.r; k += 8) {
      float gv[8], pv[8], sv[8];
      feat8<F>(g, k, gv);
      feat8<F>(ph, k, pv);
      feat8<F>(ps, k, sv);
#pragma unroll
      for (int j = 0; j < 8; ++j) delta = fmaf(gv[j] * pv[j], sv[j], delta);
    }
  }
  const float s = on ? fmaf(p.sc.alpha[i], p.cand_logit[row * K + lane], p.sc.lambda[i] * delta) : neg_inf();
  const float smax = wave_max(s);
  const float es = on ? __builtin_amdgcn_exp2f((s - smax) * kLog2e) : 0.f;
  const float ssum = wave_sum(es);
  const float lz_s = smax + __builtin_amdgcn_logf(ssum) * kLn2;  // LSE of the selector logits
  const float logq = s - lz_s;
  const float qt = on ? es / ssum : 0.f;

  const T* zr = static_cast<const T*>(p.target) + b * p.t_stride_b + i * p.t_stride_i;
  const float z = on ? logit_at<T>(zr, c) : neg_inf();
  float pt, logp;
  if (p.inv_T > 0.f) {
    const float x = on ? z * p.inv_T : neg_inf();
    const float xmax = wave_max(x);
    const float ex = on ? __builtin_amdgcn_exp2f((x - xmax) * kLog2e) : 0.f;
    const float xsum = wave_sum(ex);
    pt = on ? ex / xsum : 0.f;
    logp = x - (xmax + __builtin_amdgcn_logf(xsum) * kLn2);
  } else {
    const float zmax = wave_max(z);
    const bool top = on && z == zmax;
    const int ties = popc(ballot(top));
    pt = top ? 1.f / static_cast<float>(ties) : 0.f;
    logp = top ? -__builtin_amdgcn_logf(static_cast<float>(ties)) * kLn2 : 0.f;
  }
  const float kl = wave_sum(pt > 0.f ? pt * (logp - logq) : 0.f);

  const T* ur = static_cast<const T*>(p.logits) + b * p.stride_b + i * p.stride_i;
  const float ce = p.lse[row] - logit_at<T>(ur, y);
  const float gs = qt - pt;
  if (lane == 0) {
    p.loss[row] = kl + p.beta * ce;
    if (p.kl) p.kl[row] = kl;
    if (p.ce) p.ce[row] = ce;
  }
  if (on && p.grad_s) p.grad_s[row * K + lane] = gs;
  if (p.grad) {
    float* gr = p.grad + row * p.V;
    const bool y_in = ballot(cin && cid == y) != 0;
    if (cin) gr[c] += p.sc.alpha[i] * gs - (cid == y ? p.beta : 0.f);
    if (!y_in && lane == 0) gr[y] -= p.beta;
  }
}

template <typename T, typename F>
void launch_typed(const LossArgs& p, int rows, bool vec, hipStream_t stream) {
  if (p.grad) {
    constexpr int64_t kChunk = static_cast<int64_t>(kDenseThreads) * 8 * kDenseUnroll;
    const dim3 grid(static_cast<unsigned>(rows), static_cast<unsigned>((p.V + kChunk - 1) / kChunk));
    const T* u = static_cast<const T*>(p.logits);
    if (vec)
      hipLaunchKernelGGL((kl_dense_kernel<T, true>), grid, dim3(kDenseThreads), 0, stream, u, p.gamma, p.V,
                         p.stride_b, p.stride_i, p.lse, p.y_star, p.beta, p.grad);
    else
      hipLaunchKernelGGL((kl_dense_kernel<T, false>), grid, dim3(kDenseThreads), 0, stream, u, p.gamma, p.V,
                         p.stride_b, p.stride_i, p.lse, p.y_star, p.beta, p.grad);
  }
  hipLaunchKernelGGL((kl_position_kernel<T, F>), dim3(static_cast<unsigned>(rows)), dim3(kWave), 0, stream, p);
}

}  // namespace

hipError_t launch_tree_kl_loss(const TreeKlArgs& a, hipStream_t stream) {
  LossArgs p{};
  p.logits = a.logits;
  p.target = a.target;
  p.gamma = a.gamma;
  p.K = a.K;
  p.r = a.r;
  p.V = a.V;
  p.stride_b = a.stride_b;
  p.stride_i = a.stride_i;
  p.t_stride_b = a.t_stride_b;
  p.t_stride_i = a.t_stride_i;
  p.lse = a.lse;
  p.cand_ids = a.cand_ids;
  p.cand_logit = a.cand_logit;
  p.y_star = a.y_star;
  p.anchor = a.anchor;
  p.phi = a.phi;
  p.psi = a.psi;
  p.gate = a.gate;
  p.sc = a.sc;
  p.inv_T = a.T > 0.f ? 1.f / a.T : 0.f;
  p.beta = a.beta;
  p.loss = a.loss;
  p.kl = a.kl;
  p.ce = a.ce;
  p.grad_s = a.grad_s;
  p.grad = a.grad;
  const int rows = a.B * a.gamma;
  if (a.dtype == 1) {
    if (a.feat_dtype == 1)
      launch_typed<uint16_t, uint16_t>(p, rows, a.vec, stream);
    else
      launch_typed<uint16_t, float>(p, rows, a.vec, stream);
  } else {
    if (a.feat_dtype == 1)
      launch_typed<float, uint16_t>(p, rows, a.vec, stream);
    else
      launch_typed<float, float>(p, rows, a.vec, stream);
  }
  return hipGetLastError();
}

}  // namespace ubt
