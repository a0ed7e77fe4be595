// Head allocation units (Sec. 3, Allocation units): when decay and output
// normalisation are per head (Gated DeltaNet), every head has one width and
// FP16 scales per block of 32 key channels (rows) of each column; R~ = 1, so
// the widths follow decay alone, and b_min = 2.
//
// The column layout of the recurrence fits this format: wave w owns rows
// [32w, 32w + 32), which is exactly one scale block, and lane l owns columns
// l + 64c, so every scale group (block, column) sits in one lane's
// registers.  A lane fits its groups alone (the row quantiser's 16 clip
// factors, error in row order), and with one width b per head the block's
// 32 codes of a column are 32 b bits = b whole words of the column's bit
// stream (row i starts at bit i b), so a lane packs and stores them with no
// cross-lane traffic.
//
// A write-back runs two kernels: k_head_weights (EMA rates per row, the
// head's key = mean Gamma of its rows) and k_head_step (the head's width
// from the keys of all heads of its sequence, then load, recurrence over the
// interval's tokens with outputs, fit, pack, metadata).  The widths depend
// on the statistics only, so the allocation needs no pass over the states.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kda_device.hpp"
#include "kda_kernels.hpp"
#include "kda_profile.hpp"
#include "kda_record.hpp"
#include "kda_recur.hpp"

namespace kda {

namespace {

// Key of allocation slot (unit, level l) as in the row allocator: the
// frexp exponent of c minus 2l and the mantissa; zero keys order last.
struct SlotKey {
  int e;
  double m;
};

__device__ __forceinline__ SlotKey slot_key(double c, int l) {
  if (!(c > 0.0)) return {-0x3fffffff, 0.0};
  int e;
  const double m = frexp(c, &e);
  return {e - 2 * l, m};
}

// (a, unit ua, level la) is granted before (b, ub, lb)
__device__ __forceinline__ bool before(SlotKey a, int ua, int la, SlotKey b, int ub, int lb) {
  if (a.e != b.e) return a.e > b.e;
  if (a.m != b.m) return a.m > b.m;
  if (ua != ub) return ua < ub;
  return la < lb;
}

}  // namespace

// EMA rates of one write-back interval (tokens [tok0, tok0 + ntk)) per row
// and the head's key c_h = (sum_i Gamma_i) / d_k, rows summed in order.
template <int DK, bool BF16>
__global__ void __launch_bounds__(DK) k_head_weights(KParams p) {
  const int bh = blockIdx.x, t = threadIdx.x;
  const int b = bh / p.H, h = bh % p.H;
  const Layout L = p.L;
  const uint8_t* rec = (const uint8_t*)p.records + (long long)bh * L.slot;
  __shared__ double gam[DK];
  const unsigned ntok = *(const unsigned*)rec;
  bool fresh = ntok == 0;
  double m_run = 0.0, e_run = 0.0;
  if (!fresh) {
    m_run = exp(-2.0 * logq_decode(((const uint16_t*)(rec + L.z_off))[t]));
    e_run = 2.0 * (double)f16_to_f32(((const uint16_t*)(rec + L.r_off))[t]);
  }
  const bool erase = !p.no_erase;
  for (int j = 0; j < p.ntk; ++j) {
    const size_t th = ((size_t)b * p.T + p.tok0 + j) * p.H + h;
    const float s = p.per_head ? p.s[th] : p.s[th * DK + t];
    const double zs = decay_sample(s);
    const double ys = erase ? erase_sample(in_f32<BF16>(p.k, th * DK + t), p.beta[th]) : 0.0;
    if (fresh) {
      m_run = zs;
      e_run = ys;
    } else {
      m_run = p.one_minus_alpha * m_run + p.alpha * zs;
      e_run = p.one_minus_alpha * e_run + p.alpha * ys;
    }
    fresh = false;
  }
  const double s_hat = -0.5 * log(m_run);
  const double r = 0.5 * e_run;
  gam[t] = p.gamma ? p.gamma[(size_t)bh * DK + t] : mode_gamma(p.weight_mode, s_hat, r, p.wb_C);
  p.ws_zr[(size_t)bh * DK + t] = (uint32_t)logq_encode(s_hat) | ((uint32_t)r_encode(r) << 16);
  __syncthreads();
  if (t == 0) {
    double acc = 0.0;
    for (int i = 0; i < DK; ++i) acc = acc + gam[i];
    p.ws_c[bh] = acc / (double)DK;
  }
}

// Decode this lane's columns of the wave's 32-row block from a width-B
// record: b whole words per column.
template <int B, int CPL>
__device__ __forceinline__ void load_block(const uint32_t* codes, int dv, int w, int lane,
                                           const float (&scl)[CPL], float (&X)[ROW_BLOCK][CPL]) {
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int col = lane + WAVE * c;
    uint32_t wd[B + 1];
#pragma unroll
    for (int k = 0; k < B; ++k) wd[k] = codes[(size_t)(w * B + k) * dv + col];
    wd[B] = 0u;
#pragma unroll
    for (int r = 0; r < ROW_BLOCK; ++r) {
      const int pos = r * B, k = pos >> 5, sh = pos & 31;
      const uint32_t f = __builtin_amdgcn_alignbit(wd[k + 1], wd[k], (uint32_t)sh);
      const int code = __builtin_amdgcn_sbfe((int)f, 0, B);
      X[r][c] = (float)code * scl[c];
    }
  }
}

// Fit column c of the block (the row quantiser's candidates, error in row
// order, smallest clip factor among equal errors), pack its codes into B
// words and store them with the block scale.  Returns the number of
// candidates evaluated.
template <int B, int CPL>
__device__ __forceinline__ int fit_pack_block(const float (&X)[ROW_BLOCK][CPL], int c,
                                               const float* phi, uint32_t* codes, int dv, int w,
                                               int col, uint16_t* scale_out) {
  constexpr int n = (1 << (B - 1)) - 1;
  const float nf = (float)n;
  float mx = 0.f;
#pragma unroll
  for (int r = 0; r < ROW_BLOCK; ++r) mx = fmaxf(mx, fabsf(X[r][c]));
  float best = __builtin_inff();
  int mb = N_FIT - 1, evals = 0;
  for (int m = N_FIT - 1; m >= 0; --m) {
    const float d = f16_to_f32(f32_to_f16_sat_nonneg(mx * phi[m]));
    // the row maximum's clip error bounds this and every smaller factor
    const float emax = __builtin_fmaf(-nf, d, mx);
    if (emax >= 0.f && emax * emax > best) break;
    ++evals;
    const float inv = recip_f16_value(d);
    float err = 0.f;
#pragma unroll
    for (int r = 0; r < ROW_BLOCK; ++r) {
      const float q = __builtin_amdgcn_fmed3f(__builtin_rintf(X[r][c] * inv), -nf, nf);
      const float e = __builtin_fmaf(-q, d, X[r][c]);
      err = __builtin_fmaf(e, e, err);
    }
    if (err <= best) {
      best = err;
      mb = m;
    }
  }
  const uint16_t dh = f32_to_f16_sat_nonneg(mx * phi[mb]);
  const float d = f16_to_f32(dh);
  const float inv = recip_f16_value(d);
  uint32_t wd[B + 1];
#pragma unroll
  for (int k = 0; k <= B; ++k) wd[k] = 0u;
#pragma unroll
  for (int r = 0; r < ROW_BLOCK; ++r) {
    const int q = (int)__builtin_amdgcn_fmed3f(__builtin_rintf(X[r][c] * inv), -nf, nf);
    const uint32_t field = (uint32_t)q & ((1u << B) - 1u);
    const int pos = r * B, k = pos >> 5, sh = pos & 31;
    wd[k] |= field << sh;
    if (sh + B > 32) wd[k + 1] |= field >> (32 - sh);
  }
#pragma unroll
  for (int k = 0; k < B; ++k) codes[(size_t)(w * B + k) * dv + col] = wd[k];
  *scale_out = dh;
  return evals;
}

// All of this lane's columns of the wave's block at width B.
template <int B, int CPL>
__device__ __forceinline__ int fit_pack_cols(const float (&X)[ROW_BLOCK][CPL], const float* phi,
                                             uint32_t* codes, int dv, int w, int lane,
                                             uint16_t* bscale) {
  int evals = 0;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int col = lane + WAVE * c;
    evals += fit_pack_block<B, CPL>(X, c, phi, codes, dv, w, col, bscale + w * dv + col);
  }
  return evals;
}

constexpr int MAX_LEVELS = 6;   // b_max - b_min for head units (widths 2..8)

template <int DK>
struct HeadStepSmem {
  RowSmem<DK> rs;
  RecSmem<DK, DK> rsm;
  int rank[MAX_LEVELS];
  int width;
};

// One write-back interval of one head: tokens [p.tok0, p.tok0 + p.ntk).
template <int DK, bool BF16>
__global__ void __launch_bounds__(2 * DK) k_head_step(KParams p) {
  constexpr int DV = DK, CPL = DV / WAVE;
  const int bh = blockIdx.x, t = threadIdx.x, w = t / WAVE, lane = lane_id();
  const int b = bh / p.H, h = bh % p.H;
  const Layout L = p.L;
  uint8_t* rec = (uint8_t*)p.records + (long long)bh * L.slot;
  uint32_t* codes = (uint32_t*)(rec + L.codes_off);
  uint16_t* bscale = (uint16_t*)(rec + L.sc_off);
  __shared__ HeadStepSmem<DK> sm;

  // this head's width: its slots (h, l) ranked against the slots (u, l2) of
  // all heads of the sequence, the `need` best granted (ties to the lower
  // unit, then level).  Every thread takes a share of the comparisons and
  // counts, per slot l of this head, the slots ranked before it.
  {
    const int nl = p.bmax - p.bmin;   // at most MAX_LEVELS
    if (t < MAX_LEVELS) sm.rank[t] = 0;
    __syncthreads();
    const double* cs = p.ws_c + (size_t)b * p.H;
    const double cme = cs[h];
    const int per_l = p.H * nl;
    int cnt[MAX_LEVELS];
#pragma unroll
    for (int li = 0; li < MAX_LEVELS; ++li) cnt[li] = 0;
    for (int q = t; q < nl * per_l; q += blockDim.x) {
      const int li = q / per_l, rest = q % per_l;
      const int u = rest / nl, l2 = p.bmin + 1 + rest % nl, l = p.bmin + 1 + li;
      const bool bf = before(slot_key(cs[u], l2), u, l2, slot_key(cme, l), h, l);
#pragma unroll
      for (int k = 0; k < MAX_LEVELS; ++k) cnt[k] += (bf && k == li) ? 1 : 0;
    }
#pragma unroll
    for (int k = 0; k < MAX_LEVELS; ++k) {
      const int tot = wave_reduce_i(cnt[k], [](int x, int y) { return x + y; });
      if (lane == 0 && tot != 0) atomicAdd(&sm.rank[k], tot);
    }
    __syncthreads();
    if (t == 0) {
      int g = 0;
      for (int k = 0; k < nl; ++k) g += sm.rank[k] < p.need ? 1 : 0;
      sm.width = p.bmin + g;
    }
  }

  // the stored state of this lane's columns of the wave's block
  const unsigned ntok = *(const unsigned*)rec;
  const int wold = (int)*(const unsigned*)(rec + L.w_off);
  float X[ROW_BLOCK][CPL];
  {
    float scl[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) scl[c] = f16_to_f32(bscale[w * DV + lane + WAVE * c]);
    // a width above b_max (never written by this library) would address
    // words past the slot's capacity: such a record decodes as zero
    switch (ntok == 0 || wold > p.bmax ? 0 : wold) {
      case 2: load_block<2, CPL>(codes, DV, w, lane, scl, X); break;
      case 3: load_block<3, CPL>(codes, DV, w, lane, scl, X); break;
      case 4: load_block<4, CPL>(codes, DV, w, lane, scl, X); break;
      case 5: load_block<5, CPL>(codes, DV, w, lane, scl, X); break;
      case 6: load_block<6, CPL>(codes, DV, w, lane, scl, X); break;
      case 7: load_block<7, CPL>(codes, DV, w, lane, scl, X); break;
      case 8: load_block<8, CPL>(codes, DV, w, lane, scl, X); break;
      default:
#pragma unroll
        for (int r = 0; r < ROW_BLOCK; ++r)
#pragma unroll
          for (int c = 0; c < CPL; ++c) X[r][c] = 0.f;
    }
  }
  for (int j = 0; j < p.ntk; ++j) {
    const int tok = p.tok0 + j;
    __syncthreads();   // the previous token's readers of the row scalars are done
    load_rows<DK, BF16>(sm.rs, p, bh, tok);
    __syncthreads();
    const size_t th = ((size_t)b * p.T + tok) * p.H + h;
    recur_token<DK, DV, BF16>(X, sm.rs, sm.rsm, p.v, th * DV, p.o + th * DV, !p.no_erase);
  }
  __syncthreads();   // every read of the old record and of sm.width is ordered before the writes
  const int wn = sm.width;
  int evals;
  switch (wn) {
    case 2: evals = fit_pack_cols<2, CPL>(X, p.phi[2], codes, DV, w, lane, bscale); break;
    case 3: evals = fit_pack_cols<3, CPL>(X, p.phi[3], codes, DV, w, lane, bscale); break;
    case 4: evals = fit_pack_cols<4, CPL>(X, p.phi[4], codes, DV, w, lane, bscale); break;
    case 5: evals = fit_pack_cols<5, CPL>(X, p.phi[5], codes, DV, w, lane, bscale); break;
    case 6: evals = fit_pack_cols<6, CPL>(X, p.phi[6], codes, DV, w, lane, bscale); break;
    case 7: evals = fit_pack_cols<7, CPL>(X, p.phi[7], codes, DV, w, lane, bscale); break;
    default: evals = fit_pack_cols<8, CPL>(X, p.phi[8], codes, DV, w, lane, bscale); break;
  }
  if (p.diag_fit != nullptr) {
    // profiling: candidate evaluations of the block fits (one block-column per lane and column)
    const int tot = wave_reduce_i(evals, [](int a, int c) { return a + c; });
    if (lane == 0) atomicAdd(p.diag_fit, (unsigned long long)tot);
  }
  if (t < DK) {
    const uint32_t zr = p.ws_zr[(size_t)bh * DK + t];
    ((uint16_t*)(rec + L.z_off))[t] = (uint16_t)(zr & 0xFFFFu);
    ((uint16_t*)(rec + L.r_off))[t] = (uint16_t)(zr >> 16);
  }
  if (t == 0) {
    *(unsigned*)rec = ntok + (unsigned)p.ntk;
    *(unsigned*)(rec + L.w_off) = (unsigned)wn;
  }
}

template <int DK>
static hipError_t head_interval(const KParams& p, hipStream_t st) {
  const int nbh = p.B * p.H;
  hipError_t e = p.in_bf16 ? launch("weights", k_head_weights<DK, true>, nbh, DK, 0, st, p)
                           : launch("weights", k_head_weights<DK, false>, nbh, DK, 0, st, p);
  if (e != hipSuccess) return e;
  return p.in_bf16 ? launch("step", k_head_step<DK, true>, nbh, 2 * DK, 0, st, p)
                   : launch("step", k_head_step<DK, false>, nbh, 2 * DK, 0, st, p);
}

static hipError_t head_interval_any(const KParams& p, hipStream_t st) {
  if (p.dk == 64) return head_interval<64>(p, st);
  if (p.dk == 256) return head_interval<256>(p, st);
  return head_interval<128>(p, st);
}

hipError_t launch_step_heads(KParams p, hipStream_t st) {
  p.tok0 = 0;
  p.ntk = 1;
  return head_interval_any(p, st);
}

hipError_t launch_prefill_heads(KParams p, int C, hipStream_t st) {
  for (int t0 = 0; t0 < p.T; t0 += C) {
    p.tok0 = t0;
    p.ntk = (p.T - t0) < C ? (p.T - t0) : C;
    const hipError_t e = head_interval_any(p, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace kda
