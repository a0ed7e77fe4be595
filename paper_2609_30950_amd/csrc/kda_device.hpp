// Device-side building blocks of libkda (gfx950, wave64).
//
// Arithmetic follows the float32 contract of the method's write-back
// (see include/kda.h): every rounding below is deliberate, fused multiply-adds
// are explicit (__builtin_fmaf) and the library is built with
// -ffp-contract=off so the compiler adds none of its own.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kda {

constexpr int WAVE = 64;
constexpr int ROW_BLOCK = 32;   // rows per sequential fma chain (one wave)
constexpr int SEG = 64;         // columns per sequential error chain
constexpr int N_FIT = 16;       // clip factors f = (5 + m) / 20
constexpr int MAX_B = 16;

// Record layout of one (sequence, head) slot; identical on host and device.
struct Layout {
  int w_off, sc_off, z_off, r_off, meta_end, codes_off, wc;
  long long slot;
};

__host__ __device__ inline int round_up(int x, int a) { return (x + a - 1) / a * a; }

__host__ __device__ inline Layout make_layout(int dk, int dv, int bmax) {
  Layout L;
  L.w_off = 16;
  L.sc_off = L.w_off + dk / 2;
  L.z_off = L.sc_off + 2 * dk;
  L.r_off = L.z_off + 2 * dk;
  L.meta_end = L.r_off + 2 * dk;
  L.codes_off = round_up(L.meta_end, 256);
  L.wc = (dk * bmax + 31) / 32;
  L.slot = round_up(L.codes_off + L.wc * dv * 4, 256);
  return L;
}

// ---------------------------------------------------------------- FP16 ---
// float -> FP16 bits, round to nearest even (v_cvt_f16_f32), saturating
// at the largest finite value 65504 (0x7BFF) instead of overflowing to inf.
// The empty asm pins x as a rounded float32: without it the compiler fuses a
// preceding float multiply with this conversion into v_fma_mix*_f16, which
// rounds the exact product to FP16 once instead of rounding it to float32
// first, and so differs on FP16 midpoints.
__device__ inline uint16_t f32_to_f16_sat(float x) {
  asm volatile("" : "+v"(x));
  _Float16 h = (_Float16)x;
  uint16_t u = __builtin_bit_cast(uint16_t, h);
  if ((u & 0x7FFFu) == 0x7C00u && __builtin_isfinite(x)) u = (u & 0x8000u) | 0x7BFFu;
  return u;
}

__device__ inline float f16_to_f32(uint16_t u) {
  return (float)__builtin_bit_cast(_Float16, u);
}

// ----------------------------------------------------- wave primitives ---
__device__ inline int lane_id() { return __lane_id(); }

__device__ inline float wave_max(float v) {
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
  return v;
}

template <typename T>
__device__ inline T wave_sum(T v) {
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}

template <typename T>
__device__ inline T wave_min_t(T v) {
  for (int o = 32; o >= 1; o >>= 1) {
    T w = __shfl_xor(v, o, WAVE);
    v = w < v ? w : v;
  }
  return v;
}

template <typename T>
__device__ inline T wave_max_t(T v) {
  for (int o = 32; o >= 1; o >>= 1) {
    T w = __shfl_xor(v, o, WAVE);
    v = w > v ? w : v;
  }
  return v;
}

// inclusive prefix sum over the wave
__device__ inline int wave_incl_scan(int v) {
  const int l = lane_id();
  for (int o = 1; o < WAVE; o <<= 1) {
    int w = __shfl_up(v, o, WAVE);
    if (l >= o) v += w;
  }
  return v;
}

// Block-wide reductions through a small shared scratch of one slot per wave.
// Every thread of the block must call them; all receive the result.
template <typename T, typename Op>
__device__ inline T block_reduce(T v, T* scratch, Op op) {
  const int w = threadIdx.x / WAVE, nw = (blockDim.x + WAVE - 1) / WAVE;
  for (int o = 32; o >= 1; o >>= 1) v = op(v, __shfl_xor(v, o, WAVE));
  __syncthreads();
  if (lane_id() == 0) scratch[w] = v;
  __syncthreads();
  T r = scratch[0];
  for (int i = 1; i < nw; ++i) r = op(r, scratch[i]);
  return r;
}

// ------------------------------------------------ EMA and rate coding ---
// Statistics of the decay/erase rates kept per row (float64, token-sequential).
constexpr double LOGQ_LO = -20.0;
constexpr double LOGQ_HI = 5.0;
constexpr double LOGQ_LEVELS = 65535.0;

__device__ inline double decay_sample(float s) { return exp(-2.0 * (double)s); }

__device__ inline double erase_sample(float k, float beta) {
  const double b = (double)beta, kk = (double)k;
  return (b * (2.0 - b)) * (kk * kk);
}

__device__ inline uint16_t logq_encode(double s_hat) {
  if (!(s_hat > 0.0)) return 0;
  const double inv_step = LOGQ_LEVELS / (LOGQ_HI - LOGQ_LO);
  double u = (log2(s_hat) - LOGQ_LO) * inv_step;
  if (u != u) return 0;
  u = rint(u);
  u = u < 0.0 ? 0.0 : (u > LOGQ_LEVELS ? LOGQ_LEVELS : u);
  return (uint16_t)u;
}

__device__ inline double logq_decode(uint16_t z) {
  const double step = (LOGQ_HI - LOGQ_LO) / LOGQ_LEVELS;
  return exp2((double)z * step + LOGQ_LO);
}

__device__ inline uint16_t r_encode(double r) { return f32_to_f16_sat((float)r); }

__device__ inline double gamma_hat(double s_hat, double r) {
  double t = s_hat + r;
  t = t < 1e-12 ? 1e-12 : t;
  return 1.0 / expm1(2.0 * t);
}

}  // namespace kda
