// Gramian row weights of eq. gram (Sec. 2, Prop. 1) over a window of W
// tokens: the diagonal-erase estimate (one thread per row, sequential in time)
// and the exact matrix recursion with the full KDA transition, the reference
// the paper compares its estimate with.  Float64.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kda_device.hpp"
#include "kda_kernels.hpp"
#include "kda_profile.hpp"

namespace kda {

// Windowed Gramian weights: one thread per (b, h, row), sequential in time.
__global__ void k_window_gamma(int B, int W, int H, int DKr, int C, int per_head, int no_erase,
                               const float* q, const float* s, const float* beta,
                               const float* k, double* gamma) {
  const long long id = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long total = (long long)B * H * DKr;
  if (id >= total) return;
  const int i = (int)(id % DKr);
  const int h = (int)((id / DKr) % H);
  const int b = (int)(id / ((long long)DKr * H));
  double A = 0.0, acc = 0.0;
  for (int t = 0; t < W; ++t) {
    const size_t tok = ((size_t)b * W + t) * H + h;
    const float sv = per_head ? s[tok] : s[tok * DKr + i];
    const double y = no_erase ? 0.0 : erase_sample(k[tok * DKr + i], beta[tok]);
    const double lam = exp(-2.0 * (double)sv - y);
    if (t >= 1) {
      const double chi = (t % C == 0) ? 1.0 : 0.0;  // write-back after token t-1
      A = lam * (chi + A);
      const double qq = (double)q[tok * DKr + i];
      acc = acc + (qq * qq) * A;
    }
  }
  gamma[id] = acc / (double)W;
}

// Exact Gramian weights (eq. gram with the full transition
// F_t = (I - beta_t k_t k_t^T) diag(exp(-s_t)), the KDA erase): per head,
// backward over a window of W tokens,
//   M <- F_t^T (q_t q_t^T + M) F_t   for t = W-1 down to 1,
//   Gamma_i = (1/W) sum_t chi_{t-1} M_ii,
// chi_tau = 1 when a write-back follows token tau.  (I - beta k k^T) is
// symmetric, so with X = q q^T + M, u = X k and c = k^T u,
//   F^T X F = D (X - (beta k) u^T + (beta^2 c k - beta u) k^T) D
// (the two rank-one terms of the expansion merge), O(d_k^2) per token.
// Float64.  One block per head; thread t holds columns
// [32 (t % TPR), 32 (t % TPR) + 32) of row t / TPR (TPR = d_k / 32 threads per
// row; d_k <= 128, so the block has at most 512 threads).  The diagonal is
// followed by the row's first thread in a scalar that goes through the same
// operations as the matrix entry (r, r).
template <int DK>
__global__ void __launch_bounds__(DK * (DK / 32)) k_exact_gamma(int W, int H, int C, int per_head,
                                                               int no_erase,
                                                               const float* q, const float* s,
                                                               const float* beta, const float* k,
                                                               double* gamma) {
  constexpr int EPT = 32;
  constexpr int TPR = DK / EPT;
  constexpr int NT = DK * TPR;
  constexpr int NW = (NT + WAVE - 1) / WAVE;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int t = threadIdx.x, r = t / TPR, c0 = (t % TPR) * EPT;
  const int w = t / WAVE, lane = lane_id();
  const bool first = (t % TPR) == 0;
  __shared__ double qv[DK], kv[DK], dv[DK], uv[DK];
  __shared__ double part[NW];
  double M[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j) M[j] = 0.0;
  double mrr = 0.0, acc = 0.0;
  for (int tt = W - 1; tt >= 1; --tt) {
    const size_t tok = ((size_t)b * W + tt) * H + h;
    __syncthreads();   // the previous token's readers are done
    if (t < DK) {
      qv[t] = (double)q[tok * DK + t];
      kv[t] = (double)k[tok * DK + t];
      dv[t] = exp(-(double)(per_head ? s[tok] : s[tok * DK + t]));
    }
    const double bt = no_erase ? 0.0 : (double)beta[tok];   // no erasure: F = D
    __syncthreads();
    const double qr = qv[r], kr = kv[r], dr = dv[r];
    // X = q q^T + M and this thread's part of u_r = (X k)_r
    double ur = 0.0;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      M[j] = __builtin_fma(qr, qv[c0 + j], M[j]);
      ur = __builtin_fma(M[j], kv[c0 + j], ur);
      if (j % 4 == 3) asm volatile("" ::: "memory");   // keep LDS reads near their use
    }
    if constexpr (TPR >= 2) ur += __shfl_xor(ur, 1);
    if constexpr (TPR >= 4) ur += __shfl_xor(ur, 2);
    static_assert(TPR <= 4, "threads per row");
    // c = k^T u: one term per row, summed per wave, then over waves
    double ct = first ? kr * ur : 0.0;
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) ct += __shfl_xor(ct, o);
    if (first) uv[r] = ur;
    if (lane == 0) part[w] = ct;
    __syncthreads();
    double cc = 0.0;
#pragma unroll
    for (int i = 0; i < NW; ++i) cc += part[i];
    const double ar = bt * kr;
    const double fr = bt * bt * cc * kr - bt * ur;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      M[j] = __builtin_fma(-ar, uv[c0 + j], M[j]);
      M[j] = __builtin_fma(fr, kv[c0 + j], M[j]);
      M[j] = M[j] * (dr * dv[c0 + j]);
      if (j % 4 == 3) asm volatile("" ::: "memory");
    }
    if (first) {
      mrr = __builtin_fma(qr, qr, mrr);
      mrr = __builtin_fma(-ar, ur, mrr);
      mrr = __builtin_fma(fr, kr, mrr);
      mrr = mrr * (dr * dr);
      if (tt % C == 0) acc += mrr;   // a write-back follows token tt - 1
    }
  }
  if (first) gamma[(size_t)bh * DK + r] = acc / (double)W;
}

hipError_t launch_exact_gamma(const KParams& p, int W, int C, const float* q, const float* s,
                              const float* beta, const float* k, double* gamma, hipStream_t st) {
  const int nbh = p.B * p.H;
  if (p.dk == 64)
    return launch("weights", k_exact_gamma<64>, nbh, 128, 0, st, W, p.H, C, p.per_head,
                  p.no_erase, q, s, beta, k, gamma);
  return launch("weights", k_exact_gamma<128>, nbh, 512, 0, st, W, p.H, C, p.per_head, p.no_erase,
                q, s, beta, k, gamma);
}

hipError_t launch_window_gamma(const KParams& p, int W, int C, const float* q, const float* s,
                               const float* beta, const float* k, double* gamma, hipStream_t st) {
  const long long total = (long long)p.B * p.H * p.dk;
  const int bs = 256;
  return launch("weights", k_window_gamma, (unsigned)((total + bs - 1) / bs), bs, 0, st, p.B, W,
                p.H, p.dk, C, p.per_head, p.no_erase, q, s, beta, k, gamma);
}

}  // namespace kda
