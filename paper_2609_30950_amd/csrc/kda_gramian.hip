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
// Float64.  One block per head; thread t holds the 4 x 8 tile of M at rows
// 4 (t / G), columns 8 (t % G), G = d_k / 8 threads per row group (adjacent
// lanes of one wave), so each token's vectors are read from LDS once per
// tile row or column rather than once per element.  u is summed over the G
// tiles of a row by DPP pairings (every lane of the row ends with the same
// value); the thread whose tile holds the diagonal of its
// rows accumulates Gamma from it.
constexpr int XG_RT = 4;   // tile rows
constexpr int XG_CT = 8;   // tile columns

template <int DK>
constexpr int exact_gamma_threads() { return (DK / XG_RT) * (DK / XG_CT); }

template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const long long u = __builtin_bit_cast(long long, v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)u, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(u >> 32), CTRL, 0xF, 0xF, false);
  return __builtin_bit_cast(double, ((long long)hi << 32) | (long long)(unsigned)lo);
}

// Sum over N = 8 or 16 adjacent lanes by DPP pairings (quad xor 1, quad
// xor 2, mirror within 8, mirror within 16): each step adds a partner's value
// and partners add the same two numbers, so every lane of the group ends with
// the same sum.
template <int N>
__device__ __forceinline__ double group_sum_d(double v) {
  static_assert(N == 8 || N == 16, "group size");
  v += dpp_d<0xB1>(v);
  v += dpp_d<0x4E>(v);
  v += dpp_d<0x141>(v);
  if constexpr (N == 16) v += dpp_d<0x140>(v);
  return v;
}

template <int DK>
__global__ void __launch_bounds__(exact_gamma_threads<DK>()) k_exact_gamma(
    int W, int H, int C, int per_head, int no_erase, const float* q, const float* s,
    const float* beta, const float* k, double* gamma) {
  constexpr int G = DK / XG_CT;
  constexpr int NT = exact_gamma_threads<DK>();
  constexpr int NW = NT / WAVE;
  static_assert((G == 8 || G == 16) && NT % WAVE == 0, "row groups within a wave");
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int t = threadIdx.x, r0 = (t / G) * XG_RT, c0 = (t % G) * XG_CT;
  const int w = t / WAVE, lane = lane_id();
  // the tile holding the diagonal of rows r0..r0+3, and where it sits in it
  const bool diag = (t % G) == r0 / XG_CT;
  const int dcol = r0 % XG_CT;   // 0 or XG_RT
  static_assert(XG_CT == 2 * XG_RT, "two tile row blocks per tile width");
  // token inputs double-buffered by token parity: writing token tt's while a
  // slower wave still reads token tt + 1's needs no barrier
  __shared__ __align__(16) double qb[2][DK], kb[2][DK], db[2][DK];
  __shared__ __align__(16) double uv[DK];
  __shared__ double part[NW];
  double M[XG_RT][XG_CT];
#pragma unroll
  for (int a = 0; a < XG_RT; ++a)
#pragma unroll
    for (int j = 0; j < XG_CT; ++j) M[a][j] = 0.0;
  // diagonal sums for both positions the diagonal can take in a tile (a
  // select between two register elements would be lowered to a memory index)
  double acc0[XG_RT] = {0.0, 0.0, 0.0, 0.0}, acc1[XG_RT] = {0.0, 0.0, 0.0, 0.0};
  // token inputs one token ahead in registers (loaded while the current token runs)
  float nq = 0.f, nk = 0.f, ns = 0.f, nb = 0.f;
  auto fetch = [&](int tt) {
    const size_t tok = ((size_t)b * W + tt) * H + h;
    if (t < DK) {
      nq = q[tok * DK + t];
      nk = k[tok * DK + t];
      ns = per_head ? s[tok] : s[tok * DK + t];
    }
    nb = beta[tok];
  };
  if (W > 1) fetch(W - 1);
  for (int tt = W - 1; tt >= 1; --tt) {
    double* qv = qb[tt & 1];
    double* kv = kb[tt & 1];
    double* dv = db[tt & 1];
    if (t < DK) {
      qv[t] = (double)nq;
      kv[t] = (double)nk;
      dv[t] = exp(-(double)ns);
    }
    const double bt = no_erase ? 0.0 : (double)nb;   // no erasure: F = D
    if (tt > 1) fetch(tt - 1);
    __syncthreads();
    double qr[XG_RT], kr[XG_RT], ur[XG_RT], kc[XG_CT];
#pragma unroll
    for (int a = 0; a < XG_RT; ++a) {
      qr[a] = qv[r0 + a];
      kr[a] = kv[r0 + a];
    }
#pragma unroll
    for (int j = 0; j < XG_CT; ++j) kc[j] = kv[c0 + j];
    // X = q q^T + M and this tile's part of u = X k
#pragma unroll
    for (int a = 0; a < XG_RT; ++a) ur[a] = 0.0;
#pragma unroll
    for (int j = 0; j < XG_CT; ++j) {
      const double qc = qv[c0 + j];
#pragma unroll
      for (int a = 0; a < XG_RT; ++a) {
        M[a][j] = __builtin_fma(qr[a], qc, M[a][j]);
        ur[a] = __builtin_fma(M[a][j], kc[j], ur[a]);
      }
    }
#pragma unroll
    for (int a = 0; a < XG_RT; ++a) ur[a] = group_sum_d<G>(ur[a]);
    // c = k^T u: the row group's first tile contributes its rows, summed over
    // the first tiles of the wave, then over waves in order
    double ct = 0.0;
    if (t % G == 0) {
#pragma unroll
      for (int a = 0; a < XG_RT; ++a) {
        ct += kr[a] * ur[a];
        uv[r0 + a] = ur[a];
      }
    }
#pragma unroll
    for (int o = G; o < WAVE; o <<= 1) ct += __shfl_xor(ct, o);
    if (lane == 0) part[w] = ct;
    __syncthreads();
    double cc = 0.0;
#pragma unroll
    for (int i = 0; i < NW; ++i) cc += part[i];
    double ar[XG_RT], fr[XG_RT], dr[XG_RT];
#pragma unroll
    for (int a = 0; a < XG_RT; ++a) {
      ar[a] = bt * kr[a];
      fr[a] = bt * bt * cc * kr[a] - bt * ur[a];
      dr[a] = dv[r0 + a];
    }
#pragma unroll
    for (int j = 0; j < XG_CT; ++j) {
      const double uc = uv[c0 + j], dc = dv[c0 + j];
#pragma unroll
      for (int a = 0; a < XG_RT; ++a) {
        M[a][j] = __builtin_fma(-ar[a], uc, M[a][j]);
        M[a][j] = __builtin_fma(fr[a], kc[j], M[a][j]);
        M[a][j] = M[a][j] * (dr[a] * dc);
      }
    }
    if (diag && tt % C == 0) {   // a write-back follows token tt - 1
#pragma unroll
      for (int a = 0; a < XG_RT; ++a) {
        acc0[a] += M[a][a];
        acc1[a] += M[a][XG_RT + a];
      }
    }
  }
  if (diag) {
#pragma unroll
    for (int a = 0; a < XG_RT; ++a)
      gamma[(size_t)bh * DK + r0 + a] = (dcol == 0 ? acc0[a] : acc1[a]) / (double)W;
  }
}

hipError_t launch_exact_gamma(const KParams& p, int W, int C, const float* q, const float* s,
                              const float* beta, const float* k, double* gamma, hipStream_t st) {
  const int nbh = p.B * p.H;
  if (p.dk == 64)
    return launch("weights", k_exact_gamma<64>, nbh, exact_gamma_threads<64>(), 0, st, W, p.H, C,
                  p.per_head, p.no_erase, q, s, beta, k, gamma);
  return launch("weights", k_exact_gamma<128>, nbh, exact_gamma_threads<128>(), 0, st, W, p.H, C,
                p.per_head, p.no_erase, q, s, beta, k, gamma);
}

hipError_t launch_window_gamma(const KParams& p, int W, int C, const float* q, const float* s,
                               const float* beta, const float* k, double* gamma, hipStream_t st) {
  const long long total = (long long)p.B * p.H * p.dk;
  const int bs = 256;
  return launch("weights", k_window_gamma, (unsigned)((total + bs - 1) / bs), bs, 0, st, p.B, W,
                p.H, p.dk, C, p.per_head, p.no_erase, q, s, beta, k, gamma);
}

}  // namespace kda
