// Host-visible launch interface between the C ABI (kda_api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kda_device.hpp"

namespace kda {

// Everything a kernel needs, passed by value.
struct KParams {
  int B, H, dk, dv, G, scope, bmin, bmax, per_head, state32;
  int no_erase;             // 1: no erasure (w = v, no erase statistic)
  int weight_mode;          // allocation-key variant (WeightMode)
  int wb_C;                 // write-back interval of the call (weight variant h^(C))
  int need;                 // granted slots per scope unit: K - N * b_min
  double alpha, one_minus_alpha;
  Layout L;
  float phi[MAX_B + 1][N_FIT];   // fl32((5 + m) / (20 n_b)), n_b = 2^(b-1) - 1
  // tensors (device).  Token inputs are [B][T][H][.] with T = 1 for decode;
  // q/k/v are float32 (decode) or bf16 bit patterns (prefill).
  void* records;
  const void *q, *k, *v;
  const float *s, *beta;
  int T;                    // tokens in the input arrays
  int tok0, ntk;            // chunk: tokens [tok0, tok0 + ntk)
  int in_bf16;              // q/k/v element type
  const double* gamma;
  float* o;
  // workspace views
  double* ws_c;
  uint32_t* ws_zr;
  uint8_t* ws_bits;
  float* ws_s32;            // float32 state after the token, [B][H][dk][dv]
  float* ws_rpart;          // prefill: row maxima per 64-column slice, [B][H][dk][dv/64]
  double* ws_gam;           // prefill: row weights Gamma, [B][H][dk]
  float* ws_hv;             // decode: token vectors per head {w[dv], a[dk], g[dk]}
  uint8_t* ws_chunk;        // chunked prefill: per-chunk records of a group of chunks
  unsigned long long* diag_fit;  // profiling: candidate evaluations (or null)
};

hipError_t launch_step(const KParams& p, hipStream_t st);
hipError_t launch_step_outputs(const KParams& p, hipStream_t st);
hipError_t launch_step_writeback(const KParams& p, hipStream_t st);
hipError_t launch_prefill(KParams p, int C, hipStream_t st);
// Allocation and requantisation of one prefill write-back from the float32
// state, per-slice row maxima (nsl per row), Gamma and rate codes in the
// workspace (keys: the allocation weights are in ws_c already).
hipError_t launch_chunk_writeback(const KParams& p, int nsl, hipStream_t st, bool keys = false);
// Chunked prefill (WY/UT form on MFMA), d_k = d_v in {64, 128}, C <= 64.
hipError_t launch_prefill_chunked(const KParams& p, int C, hipStream_t st, hipStream_t aux);
// Bytes of one chunk record (per chunk and head) and chunks per group for
// B*H heads.
size_t chunk_record_bytes(int dk);
int chunk_group(int nbh);
// Head allocation units with block scales: a decode step (C = 1) and a
// prefill with a write-back every C tokens.
hipError_t launch_step_heads(KParams p, hipStream_t st);
hipError_t launch_prefill_heads(KParams p, int C, hipStream_t st);
// Per-token decay-gate quantisation of s [B][T][H][d_k] into out.
hipError_t launch_gate_quant(const KParams& p, int T, int bits, int linear, const float* s,
                             float* out, hipStream_t st);
hipError_t launch_pack(const KParams& p, const float* S, const uint8_t* bits, const double* s_hat,
                       const double* r, unsigned ntok, hipStream_t st);
hipError_t launch_unpack(const KParams& p, float* S, uint8_t* bits, double* s_hat, double* r,
                         hipStream_t st);
hipError_t launch_alloc_bits(const KParams& p, const double* gamma, const float* R, uint8_t* bits,
                             hipStream_t st);
hipError_t launch_exact_gamma(const KParams& p, int W, int C, const float* q, const float* s,
                              const float* beta, const float* k, double* gamma, hipStream_t st);
hipError_t launch_window_gamma(const KParams& p, int W, int C, const float* q, const float* s,
                               const float* beta, const float* k, double* gamma, hipStream_t st);

}  // namespace kda
