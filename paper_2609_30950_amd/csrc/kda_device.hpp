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
constexpr int RMS_RUN = 64;     // rows per run of a group's sum of squares (runs in order)

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

// Record layout of a head allocation unit (one width per head, FP16 scales
// per block of 32 rows of one column): u32 tokens, u32 width at w_off = 4,
// 8 reserved bytes, rate codes u16[dk], erase rates FP16[dk], block scales
// FP16[dk/32][dv] at sc_off, code words at the next multiple of 256.
__host__ __device__ inline Layout make_head_layout(int dk, int dv, int bmax) {
  Layout L;
  L.w_off = 4;
  L.z_off = 16;
  L.r_off = L.z_off + 2 * dk;
  L.sc_off = L.r_off + 2 * dk;
  L.meta_end = L.sc_off + (dk / 32) * dv * 2;
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
__device__ __forceinline__ uint16_t f32_to_f16_sat(float x) {
  asm volatile("" : "+v"(x));
  _Float16 h = (_Float16)x;
  uint16_t u = __builtin_bit_cast(uint16_t, h);
  if ((u & 0x7FFFu) == 0x7C00u && __builtin_isfinite(x)) u = (u & 0x8000u) | 0x7BFFu;
  return u;
}

// FP16 bits of a non-negative float (scales R phi of the fit), round to
// nearest even, saturating at 65504: the same value as f32_to_f16_sat for
// x >= 0 with the saturation as one median of (x, 0, 65504) before the
// conversion (values from 65504 up round to 65504 either way; NaN and -0 are
// not inputs).
__device__ __forceinline__ uint16_t f32_to_f16_sat_nonneg(float x) {
  asm volatile("" : "+v"(x));
  return __builtin_bit_cast(uint16_t, (_Float16)__builtin_amdgcn_fmed3f(x, 0.0f, 65504.0f));
}

// fl32(1 / d) for d an FP16 value (positive, or 0 -> 0): the hardware
// reciprocal refined by one Newton step, fma(r0, fma(-d, r0, 1), r0), which
// equals the correctly rounded quotient for every positive finite FP16 value
// (checked exhaustively on gfx950 against the IEEE division).
__device__ __forceinline__ float recip_f16_value(float d) {
  const float r0 = __builtin_amdgcn_rcpf(d);
  const float r1 = __builtin_fmaf(r0, __builtin_fmaf(-d, r0, 1.0f), r0);
  return d > 0.f ? r1 : 0.f;
}

__device__ __forceinline__ float f16_to_f32(uint16_t u) {
  return (float)__builtin_bit_cast(_Float16, u);
}

// ----------------------------------------------------- wave primitives ---
__device__ __forceinline__ int lane_id() { return __lane_id(); }

// DPP lane exchange within 16-lane rows (quad permutes and mirrors).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Broadcast lane `l` of v to the wave (scalar register).
__device__ __forceinline__ int bcast_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ float bcast_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Maximum over the 64 lanes of a wave, returned wave-uniform.  DPP steps
// (xor 1, xor 2, half-row mirror, row mirror) leave every lane with its
// 16-lane row maximum; the four row maxima are then read as scalars.
__device__ __forceinline__ float wave_max_uniform(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));    // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_f<0x4E>(v));    // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_f<0x141>(v));   // row_half_mirror
  v = fmaxf(v, dpp_f<0x140>(v));   // row_mirror
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

// Inclusive prefix sum over the wave: Hillis-Steele within 16-lane rows
// (row shifts by 1, 2, 4, 8; lanes without a source add 0), then the row
// totals are carried across rows with row_bcast:15 and row_bcast:31.
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_add_src(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xF, false);
}

__device__ __forceinline__ int wave_incl_scan(int v) {
  v += dpp_add_src<0x111, 0xF>(v);
  v += dpp_add_src<0x112, 0xF>(v);
  v += dpp_add_src<0x114, 0xF>(v);
  v += dpp_add_src<0x118, 0xF>(v);
  v += dpp_add_src<0x142, 0xA>(v);
  v += dpp_add_src<0x143, 0xC>(v);
  return v;
}

// DPP exchange for 32-bit integers.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}

// Wave-wide reduction of a 32-bit int, returned wave-uniform: four DPP steps
// reduce within 16-lane rows, then the four row results are read as scalars.
template <typename Op>
__device__ __forceinline__ int wave_reduce_i(int v, Op op) {
  v = op(v, dpp_i<0xB1>(v));
  v = op(v, dpp_i<0x4E>(v));
  v = op(v, dpp_i<0x141>(v));
  v = op(v, dpp_i<0x140>(v));
  return op(op(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
            op(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

// Block-wide reductions of a 32-bit int through a small shared scratch of one
// slot per wave.  Every thread of the block must call them; all receive the
// result.
template <typename Op>
__device__ __forceinline__ int block_reduce(int v, int* scratch, Op op) {
  const int w = threadIdx.x / WAVE, nw = (blockDim.x + WAVE - 1) / WAVE;
  v = wave_reduce_i(v, op);
  __syncthreads();
  if (lane_id() == 0) scratch[w] = v;
  __syncthreads();
  int r = scratch[0];
  for (int i = 1; i < nw; ++i) r = op(r, scratch[i]);
  return r;
}

// Block-wide (sum, min, max) of three ints in one pass (two barriers).
__device__ __forceinline__ void block_sum_min_max(int& sum, int& mn, int& mx, int* scratch) {
  const int w = threadIdx.x / WAVE, nw = (blockDim.x + WAVE - 1) / WAVE;
  sum = wave_reduce_i(sum, [](int a, int b) { return a + b; });
  mn = wave_reduce_i(mn, [](int a, int b) { return a < b ? a : b; });
  mx = wave_reduce_i(mx, [](int a, int b) { return a > b ? a : b; });
  __syncthreads();
  if (lane_id() == 0) {
    scratch[3 * w] = sum;
    scratch[3 * w + 1] = mn;
    scratch[3 * w + 2] = mx;
  }
  __syncthreads();
  sum = scratch[0];
  mn = scratch[1];
  mx = scratch[2];
  for (int i = 1; i < nw; ++i) {
    sum += scratch[3 * i];
    mn = scratch[3 * i + 1] < mn ? scratch[3 * i + 1] : mn;
    mx = scratch[3 * i + 2] > mx ? scratch[3 * i + 2] : mx;
  }
}

// ------------------------------------------------ EMA and rate coding ---
// Statistics of the decay/erase rates kept per row (float64, token-sequential).
constexpr double LOGQ_LO = -20.0;
constexpr double LOGQ_HI = 5.0;
constexpr double LOGQ_LEVELS = 65535.0;

__device__ __forceinline__ double decay_sample(float s) { return exp(-2.0 * (double)s); }

__device__ __forceinline__ double erase_sample(float k, float beta) {
  const double b = (double)beta, kk = (double)k;
  return (b * (2.0 - b)) * (kk * kk);
}

__device__ __forceinline__ uint16_t logq_encode(double s_hat) {
  if (!(s_hat > 0.0)) return 0;
  const double inv_step = LOGQ_LEVELS / (LOGQ_HI - LOGQ_LO);
  double u = (log2(s_hat) - LOGQ_LO) * inv_step;
  if (u != u) return 0;
  u = rint(u);
  u = u < 0.0 ? 0.0 : (u > LOGQ_LEVELS ? LOGQ_LEVELS : u);
  return (uint16_t)u;
}

__device__ __forceinline__ double logq_decode(uint16_t z) {
  const double step = (LOGQ_HI - LOGQ_LO) / LOGQ_LEVELS;
  return exp2((double)z * step + LOGQ_LO);
}

__device__ __forceinline__ uint16_t r_encode(double r) { return f32_to_f16_sat((float)r); }

__device__ __forceinline__ double gamma_hat(double s_hat, double r) {
  double t = s_hat + r;
  t = t < 1e-12 ? 1e-12 : t;
  return 1.0 / expm1(2.0 * t);
}

// Allocation-key variants of the weight ablations (Sec. 5, Table ablate);
// the values of kda_config.weight_mode.
enum WeightMode {
  WM_EMA = 0,            // Gamma^ R~^2 (eq. weight)
  WM_RANGE = 1,          // R^2, raw range alone
  WM_GAMMA_RAW = 2,      // Gamma^ R^2
  WM_REL_RANGE = 3,      // R~^2
  WM_PERSIST = 4,        // w^(1) R~^2, w^(1) = 1/(1 - exp(-2 s^)) (DAMP, uncapped)
  WM_WRITEBACK = 5,      // h^(C) R~^2, h^(C) = 1/(1 - exp(-2 C s^))
  WM_NO_ERASE_RATE = 6,  // Gamma^ with r = 0, times R~^2
  WM_UNIFORM = 7,        // equal keys: uniform widths
  WM_DECAY = 8,          // Gamma^ alone (ranges ignored)
};

// Row factor of the key; rates clamped below at 1e-12 as in gamma_hat.
__device__ __forceinline__ double mode_gamma(int mode, double s_hat, double r, int C) {
  if (mode == WM_EMA || mode == WM_GAMMA_RAW || mode == WM_DECAY) return gamma_hat(s_hat, r);
  if (mode == WM_NO_ERASE_RATE) return gamma_hat(s_hat, 0.0);
  const double s = s_hat < 1e-12 ? 1e-12 : s_hat;
  if (mode == WM_PERSIST) return 1.0 / -expm1(-2.0 * s);
  if (mode == WM_WRITEBACK) return 1.0 / -expm1((-2.0 * (double)C) * s);
  return 1.0;   // range, relative range, uniform
}

// Key c of a row from its factor, row maximum and group RMS.
__device__ __forceinline__ double mode_key(int mode, double gam, float R, double rms) {
  if (mode == WM_UNIFORM) return 1.0;
  if (mode == WM_DECAY) return gam;
  if (mode == WM_RANGE || mode == WM_GAMMA_RAW) {
    const double Rr = (double)R;
    return gam * (Rr * Rr);
  }
  const double Rt = rms > 0.0 ? (double)R / rms : 0.0;
  return gam * (Rt * Rt);
}

}  // namespace kda
