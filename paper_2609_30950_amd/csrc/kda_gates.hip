// Per-token decay-gate quantisation (Sec. 3, Decay-gate quantization): the
// rates s of one (sequence, token, head) are coded with 2^b levels uniform in
// log s (or, for comparison, in g = -s) over the range of the head's channels
// at that token, and replaced by their dequantised values.  One wave per
// (sequence, token, head), d_k / 64 channels per lane, float64 arithmetic.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kda_device.hpp"
#include "kda_kernels.hpp"
#include "kda_profile.hpp"

namespace kda {

namespace {

__device__ __forceinline__ double wave_min_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmin(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ double wave_max_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmax(v, __shfl_xor(v, o));
  return v;
}

}  // namespace

template <int DK>
__global__ void __launch_bounds__(256) k_gate_quant(const float* s, float* out, long long rows,
                                                    int bits, int linear) {
  constexpr int PER = DK / WAVE;
  const long long row = (long long)blockIdx.x * 4 + threadIdx.x / WAVE;
  if (row >= rows) return;   // whole waves leave together
  const int lane = lane_id();
  const float* src = s + row * DK;
  double x[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const double v = (double)src[lane + WAVE * u];
    x[u] = linear ? v : log(v);
  }
  double lo = x[0], hi = x[0];
#pragma unroll
  for (int u = 1; u < PER; ++u) {
    lo = fmin(lo, x[u]);
    hi = fmax(hi, x[u]);
  }
  lo = wave_min_d(lo);
  hi = wave_max_d(hi);
  const double n = (double)((1 << bits) - 1);
  const double step = (hi - lo) / n;
  float* dst = out + row * DK;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    double code = 0.0;
    if (step > 0.0) code = fmin(fmax(rint((x[u] - lo) / step), 0.0), n);
    const double xh = lo + code * step;
    dst[lane + WAVE * u] = (float)(linear ? xh : exp(xh));
  }
}

hipError_t launch_gate_quant(const KParams& p, int T, int bits, int linear, const float* s,
                             float* out, hipStream_t st) {
  const long long rows = (long long)p.B * T * p.H;
  const unsigned blocks = (unsigned)((rows + 3) / 4);
  if (p.dk == 64) return launch("gates", k_gate_quant<64>, blocks, 256, 0, st, s, out, rows, bits, linear);
  if (p.dk == 256) return launch("gates", k_gate_quant<256>, blocks, 256, 0, st, s, out, rows, bits, linear);
  return launch("gates", k_gate_quant<128>, blocks, 256, 0, st, s, out, rows, bits, linear);
}

}  // namespace kda
