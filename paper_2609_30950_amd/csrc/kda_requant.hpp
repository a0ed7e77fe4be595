// Requantisation of a head's float32 state into a record (Sec. 3): widths
// ordered for the fit, the clip-factor fit of every row with its FP16 scale
// and codes, and the packing of the column bit streams, for the decode step
// (whole heads, state rebuilt from the record) and the prefill write-backs
// (from the float32 state, optionally two blocks per head).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kda_alloc.hpp"
#include "kda_device.hpp"
#include "kda_kernels.hpp"
#include "kda_record.hpp"

namespace kda {

// ----------------------------------------------------- row-layout fit ---

// Codes in LDS: int16 (widths up to 16) for d_k <= 128, int8 for d_k = 256
// (widths up to 8), so that the column-major code tile fits in LDS.
template <int DK>
using CodeT = typename std::conditional<(DK > 128), int8_t, int16_t>::type;

// Column stride (elements) of the column-major code buffer: padded by 16 bytes
// so that the 16-byte reads of consecutive columns hit distinct LDS banks.
template <int DK>
constexpr int CT_LD_OF = DK + 16 / (int)sizeof(CodeT<DK>);
template <int DK, typename CT>
constexpr int ct_ld() { return DK + 16 / (int)sizeof(CT); }

// Sum of the per-segment partials of one row held by SEGS adjacent lanes, in
// the halving order (p[s] + p[s + SEGS/2] first), via DPP quad permutes.
template <int SEGS>
__device__ __forceinline__ float seg_combine(float v) {
  static_assert(SEGS == 1 || SEGS == 2 || SEGS == 4, "segments per row");
  if constexpr (SEGS == 4) v = v + dpp_f<0x4E>(v);   // lanes differing in bit 1
  if constexpr (SEGS >= 2) v = v + dpp_f<0xB1>(v);   // lanes differing in bit 0
  return v;
}

// Order rows by width, widest first (ties by row index), so that each wave of
// the fit holds rows of similar width and similar pruning depth.  Also forms
// the prefix sums P[i] of the new widths (row bit offsets of the packed
// streams).  Wave-ballot counting; threads t < DK own row t.
template <int DK>
struct OrderSmem {
  int cnt[DK / WAVE][MAX_B + 1];
  int P[DK + 1];
};

// perm[0 .. hi - lo) lists the rows lo .. hi - 1 by width, widest first
// (ties in row order); os.P holds the bit offsets of all DK rows.  vmax: the
// largest width any row may have (the counts above it are not formed).
template <int DK>
__device__ __forceinline__ void width_order(const uint8_t* bits, uint8_t* perm, OrderSmem<DK>& os,
                                            int lo = 0, int hi = DK, int vmax = MAX_B) {
  const int t = threadIdx.x, w = t / WAVE, lane = lane_id();
  int b = 0, bp = 0, below = 0;
  if (t < DK) {
    b = bits[t];
    bp = t >= lo && t < hi ? b : 0;   // widths are at least 1: 0 marks rows outside the range
    const unsigned long long lt = (1ull << lane) - 1ull;
    for (int v = 1; v <= vmax; ++v) {
      const unsigned long long m = __ballot(bp == v);
      if (lane == 0) os.cnt[w][v] = __popcll(m);
      if (bp == v) below = __popcll(m & lt);
    }
    // prefix sums of widths in row order
    const int incl = wave_incl_scan(b);
    os.P[t + 1] = incl;          // per-wave inclusive; fixed up below
  }
  __syncthreads();
  if (bp > 0) {
    int pos = below;
    for (int v = bp + 1; v <= vmax; ++v)
      for (int q = 0; q < DK / WAVE; ++q) pos += os.cnt[q][v];
    for (int q = 0; q < w; ++q) pos += os.cnt[q][bp];
    perm[pos] = (uint8_t)t;
  }
  // wave totals of widths -> global prefix
  int carry = 0;
  if (t < DK)
    for (int q = 0; q < w; ++q) carry += os.P[(q + 1) * WAVE];
  __syncthreads();
  if (t < DK) os.P[t + 1] += carry;
  if (t == 0) os.P[0] = 0;
  __syncthreads();
}

// Sum of the per-segment partials of one row over its SEGS segment lanes,
// which sit PAIRS lanes apart (PAIRS = 2: the two candidate lanes of a
// segment are adjacent), in the halving order of seg_combine.
template <int SEGS, int PAIRS>
__device__ __forceinline__ float seg_combine_p(float v) {
  if constexpr (PAIRS == 1) {
    return seg_combine<SEGS>(v);
  } else {
    static_assert(SEGS <= 2, "candidate lanes with at most two segments per row");
    if constexpr (SEGS == 2) {
      if constexpr (PAIRS == 2) v = v + dpp_f<0x4E>(v);   // lanes differing in bit 1
      else v = v + __shfl_xor(v, PAIRS);                  // lanes differing in bit log2(PAIRS)
    }
    return v;
  }
}

// Lane q of each group of four (quad_perm [q, q, q, q]).
template <int Q>
__device__ __forceinline__ float quad_lane(float v) {
  return dpp_f<Q * 0x55>(v);
}

// Ternary rows (width 2: levels -Delta, 0, Delta).  The general evaluation
// codes x as c = clamp(rint(fl32(x inv)), -1, 1), so |c| = 1 exactly when
// fl32(|x| inv) > 1/2, i.e. when |x| > th, th the largest float with
// fl32(th inv) <= 1/2 (fl32(a inv) is monotone in a; th lies within three
// ulps of Delta / 2, which is exact).  With K = 2^(23 - E), E the exponent of
// th, K (|x| - th) is at least 1 for every float |x| > th and at most 0
// otherwise, so clamping fma(|x|, K, -K th) to [0, 1] gives |c| in one
// operation; fma(-|c|, Delta, |x|) is then +-fma(-c, Delta, x), so the error
// sum is the same float32 value.  Delta = 0 (inv = 0): no |x| passes.
__device__ __forceinline__ void ternary_threshold(float d, float inv, float& K, float& nKth) {
  if (!(d > 0.f)) {
    K = 1.f;
    nKth = -__builtin_inff();
    return;
  }
  const int a0 = __builtin_bit_cast(int, 0.5f * d);
  float th = __builtin_bit_cast(float, a0 - 3);
#pragma unroll
  for (int k = -2; k <= 3; ++k) {
    const float c = __builtin_bit_cast(float, a0 + k);
    if (c * inv <= 0.5f) th = c;
  }
  const int E = ((__builtin_bit_cast(int, th) >> 23) & 255) - 127;
  K = __builtin_bit_cast(float, (127 + 23 - E) << 23);
  nKth = -(K * th);
}

// |c| of a ternary row: fma(|x|, K, -K th) clamped to [0, 1].
__device__ __forceinline__ float ternary_code(float x, float K, float nKth) {
  return __builtin_amdgcn_fmed3f(__builtin_fmaf(fabsf(x), K, nKth), 0.f, 1.f);
}

// Quantise the rows of a row-major float32 state S[DK][DV] (device memory)
// with widths bits[] (method: see the top of this file and include/kda.h).
// Thread t handles the 64-column segment t % (DV/64) of row
// perm[t / (DV/64)].  Writes int16 codes column-major into Ct[DV][CT_LD]
// (LDS) and FP16 scales.
//
// Exact pruning: candidates are scanned from f = 1 downwards.  For m with
// n Delta_m <= R the row maximum is coded as +-n, so its squared residual
// fl(e_max^2), e_max = fl(R - n Delta_m), is a lower bound of err_m (the error
// is a float32 sum of non-negative terms that contains it), and e_max only
// grows as m falls.  Once that bound exceeds the best error no smaller f can
// reach the minimum, so the scan stops; the result equals the exhaustive
// first strict minimum over all 16 candidates.
//
// PAIRS = 2 or 4 (blocks of 2 PAIRS d_k threads, for grids with few heads):
// PAIRS adjacent lanes hold the same segment and evaluate the candidates
// m, m - 1, .., m - PAIRS + 1 of one step together.  Every bound of a step is
// tested against the best error before the step, so a candidate may be
// evaluated where the sequential scan would have stopped; its error then
// exceeds the best (the bound is a lower bound), the merge in candidate order
// passes over it and the scan ends after the step: the same choice, at most
// PAIRS - 1 evaluations more per row.
// ROWS: the rows perm[0 .. ROWS) (a block may take part of a head's rows).
template <int DK, int DV, bool SYNC_AFTER_LOAD = false, int PAIRS = 1, int ROWS = DK,
          typename LoadRow, typename CT>
__device__ __forceinline__ void fit_rows(LoadRow load_row, const uint8_t* bits, const uint8_t* perm,
                         const float (*phi)[N_FIT], CT* Ct, uint16_t* scale_out,
                         unsigned long long* diag) {
  constexpr int LD = ct_ld<DK, CT>();
  constexpr int SEGS = DV / SEG;
  constexpr int ITEMS = ROWS * SEGS * PAIRS;
  static_assert(PAIRS == 1 || PAIRS == 2 || PAIRS == 4, "candidates per step");
  static_assert(N_FIT % PAIRS == 0, "whole candidate pairs");
  const int tid = threadIdx.x, nt = blockDim.x;
  const int iters = (ITEMS + nt - 1) / nt;   // same count for every thread
  for (int rep = 0; rep < iters; ++rep) {
  const int unit = rep * nt + tid;
  const bool valid = unit < ITEMS;
  const int half = unit % PAIRS;   // this lane's candidate within a step
  const int item = unit / PAIRS;
  const int i = valid ? perm[item / SEGS] : 0;
  const int sg = item % SEGS;
  float x[SEG];
  load_row(i, sg, x);
  // the code tile may share LDS with what the loader reads (one item per thread)
  if constexpr (SYNC_AFTER_LOAD) __syncthreads();
  float mx = 0.f;
#pragma unroll
  for (int j = 0; j < SEG; ++j) mx = fmaxf(mx, fabsf(x[j]));
  if constexpr (PAIRS == 1) {
    if constexpr (SEGS >= 2) mx = fmaxf(mx, dpp_f<0xB1>(mx));
    if constexpr (SEGS >= 4) mx = fmaxf(mx, dpp_f<0x4E>(mx));
  } else if constexpr (SEGS >= 2) {
    mx = fmaxf(mx, PAIRS == 2 ? dpp_f<0x4E>(mx) : __shfl_xor(mx, PAIRS));
  }
  const int b = bits[i];
  CT* dst = Ct + (size_t)(sg * SEG) * LD + i;
  // the first lane of a candidate pair writes the codes and the scale
  const bool writer = valid && half == 0;
  int evals = 0;
  if (b == 1) {
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < SEG; ++j) acc = acc + fabsf(x[j]);
    // halving over segments: lanes differing in the top segment bit first
    acc = seg_combine_p<SEGS, PAIRS>(acc);
    const uint16_t mu = f32_to_f16_sat(acc * (1.0f / (float)DV));
    if (writer) {
#pragma unroll
      for (int j = 0; j < SEG; ++j) dst[(size_t)j * LD] = (CT)(x[j] < 0.f ? 1 : 0);
      if (sg == 0) scale_out[i] = mu;
    }
  } else {
    const float nf = (float)((1 << (b - 1)) - 1);
    float best = __builtin_inff();
    int mb = N_FIT - 1;
    if constexpr (PAIRS == 1) {
      // waves whose rows all have width 2 take the three-operation form of
      // the same evaluation (ternary_threshold)
      const bool ternary = __all(b == 2);
      // factors read through one running pointer: the read after the last
      // candidate (m = 0) lands on the previous width's last factor (b >= 2
      // here), in the table and unused
      const float* pp = &phi[0][0] + b * N_FIT + N_FIT - 1;
      float ph = *pp;
      for (int m = N_FIT - 1; m >= 0; --m) {
        const float d = f16_to_f32(f32_to_f16_sat_nonneg(mx * ph));
        ph = *--pp;   // next candidate's factor, off the critical path
        const float emax = __builtin_fmaf(-nf, d, mx);
        if (emax >= 0.f && emax * emax > best) break;   // row-uniform decision
        ++evals;
        const float inv = recip_f16_value(d);
        float err = 0.f;
        if (ternary) {
          float K, nKth;
          ternary_threshold(d, inv, K, nKth);
#pragma unroll
          for (int j = 0; j < SEG; ++j) {
            const float e = __builtin_fmaf(-ternary_code(x[j], K, nKth), d, fabsf(x[j]));
            err = __builtin_fmaf(e, e, err);
          }
        } else {
#pragma unroll
          for (int j = 0; j < SEG; ++j) {
            const float c = __builtin_amdgcn_fmed3f(__builtin_rintf(x[j] * inv), -nf, nf);
            const float e = __builtin_fmaf(-c, d, x[j]);
            err = __builtin_fmaf(e, e, err);
          }
        }
        err = seg_combine<SEGS>(err);
        if (err <= best) { best = err; mb = m; }
      }
    } else {
      for (int m0 = N_FIT - 1; m0 >= PAIRS - 1; m0 -= PAIRS) {
        // the step's candidates m0 - q, their bounds against the best so far
        float dq[PAIRS];
        bool stop[PAIRS];
#pragma unroll
        for (int q = 0; q < PAIRS; ++q) {
          dq[q] = f16_to_f32(f32_to_f16_sat_nonneg(mx * phi[b][m0 - q]));
          const float e = __builtin_fmaf(-nf, dq[q], mx);
          stop[q] = e >= 0.f && e * e > best;
        }
        if (stop[0]) break;                       // row-uniform decisions
        float d = dq[0];
        bool skip = false;
#pragma unroll
        for (int q = 1; q < PAIRS; ++q) {
          d = half == q ? dq[q] : d;
          skip = half == q ? stop[q] : skip;
        }
        if (!skip) ++evals;
        const float inv = recip_f16_value(d);
        float err = 0.f;
#pragma unroll
        for (int j = 0; j < SEG; ++j) {
          const float c = __builtin_amdgcn_fmed3f(__builtin_rintf(x[j] * inv), -nf, nf);
          const float e = __builtin_fmaf(-c, d, x[j]);
          err = __builtin_fmaf(e, e, err);
        }
        err = seg_combine_p<SEGS, PAIRS>(err);
        // every lane of the step merges the errors in candidate order
        float eq[PAIRS];
        if constexpr (PAIRS == 2) {
          const float other = dpp_f<0xB1>(err);   // the partner lane's candidate
          eq[0] = half ? other : err;
          eq[1] = half ? err : other;
        } else {
          eq[0] = quad_lane<0>(err);
          eq[1] = quad_lane<1>(err);
          eq[2] = quad_lane<2>(err);
          eq[3] = quad_lane<3>(err);
        }
        bool any = false;
#pragma unroll
        for (int q = 0; q < PAIRS; ++q) {
          if (!stop[q] && eq[q] <= best) { best = eq[q]; mb = m0 - q; }
          any = any || stop[q];
        }
        if (any) break;
      }
    }
    const uint16_t dh = f32_to_f16_sat_nonneg(mx * phi[b][mb]);
    const float d = f16_to_f32(dh);
    const float inv = recip_f16_value(d);
    if (writer) {
      // c = clamp(rint(fl32(x inv)), -n, n) as M + c, M = 1.5 2^23: adding M
      // to fl32(x inv) rounds it to an integer, ties to even, exactly as rint
      // does while |x inv| < 2^22 (larger magnitudes clamp to the same code),
      // and the low bits of M + c (a float in [2^23, 2^24)) are c in two's
      // complement, which the truncating store keeps
      constexpr float M = 12582912.0f;
      const float lo = M - nf, hi = M + nf;
#pragma unroll
      for (int j = 0; j < SEG; ++j) {
        const float c = __builtin_amdgcn_fmed3f(x[j] * inv + M, lo, hi);
        dst[(size_t)j * LD] = (CT)__builtin_bit_cast(uint32_t, c);
      }
      if (sg == 0) scale_out[i] = dh;
    }
  }
  if (diag != nullptr) {
    // all lanes have reconverged here
    const int tot = wave_reduce_i(valid ? evals : 0, [](int a, int c) { return a + c; });
    if (lane_id() == 0) atomicAdd(diag, (unsigned long long)tot);
  }
  }
}

// Pack codes Ct[DV][CT_LD] (column-major) with widths bits[] into column
// bit streams, rows [r0, r0 + ROWS) of the head (a block may take part of a
// head's rows).  Thread (column, half) packs half of those rows, starting at
// bit P of its first row; the word both halves share (if the boundary is not
// word aligned) is merged through LDS.  A wave holds one half, so the widths,
// the bit position and every word boundary are wave-uniform (scalar
// registers and branches): each code costs one field extract and one
// shift-or into the current word.  A word that holds bits of rows outside
// the range (a neighbouring block's) is written with an atomic AND that
// clears this block's bits and an atomic OR that sets them, so the two
// blocks' writes commute; words the block owns entirely are plain stores.
template <int DK, int DV, int ROWS = DK, typename CT>
__device__ __forceinline__ void pack_cols(const CT* Ct, const uint8_t* bits, const int* P,
                                          uint32_t* words, uint32_t* tail, int r0 = 0) {
  constexpr int HALF = ROWS / 2;
  static_assert(DV == DK && DV % WAVE == 0, "one (column, half) per thread, halves wave-aligned");
  const int tid = threadIdx.x;
  const int col = tid % DV;
  // threads past 2 d_v (blocks of the paired fit) only join the barrier
  const int half = __builtin_amdgcn_readfirstlane(tid / DV);
  const bool packer = half < 2;
  const int a = r0 + (packer ? half : 0) * HALF;
  const int start = __builtin_amdgcn_readfirstlane(P[a]);
  const int split = __builtin_amdgcn_readfirstlane(P[r0 + HALF]);
  // stream bits this block owns: [own_lo, own_hi); the block of the last
  // rows also owns the padding of the last word
  const int own_lo = __builtin_amdgcn_readfirstlane(P[r0]);
  const int own_hi = r0 + ROWS >= DK ? 0x7fffffff : __builtin_amdgcn_readfirstlane(P[r0 + ROWS]);
  auto put = [&](int wi, uint32_t v) {   // wi is wave-uniform
    uint32_t* dst = words + (size_t)wi * DV + col;
    const int b0 = own_lo - 32 * wi, b1 = own_hi - 32 * wi;
    if (b0 <= 0 && b1 >= 32) {
      __builtin_nontemporal_store(v, dst);   // read again only by a later step
    } else {
      const uint32_t m = (b1 >= 32 ? ~0u : (1u << b1) - 1u) & (b0 <= 0 ? ~0u : ~((1u << b0) - 1u));
      atomicAnd(dst, ~m);
      atomicOr(dst, v & m);
    }
  };
  // widths, four per LDS word (bits[] is 4-byte aligned), read as broadcasts
  const uint32_t* bw = (const uint32_t*)(bits + a);
  uint32_t cur = 0;         // bits [32 wi, 32 wi + nb) of this column's stream
  int nb = start & 31;      // bits below nb in the first word belong to earlier rows
  int wi = start >> 5;
  uint32_t first = 0;       // upper half: its first word, merged after the barrier
  bool first_pending = half == 1 && (split & 31) != 0;
  constexpr int CB = (int)sizeof(CT);   // bytes per code
  constexpr int CPR = 16 / CB;                  // codes per 16-byte read
  static_assert(HALF % CPR == 0, "whole 16-byte code reads per half");
  const CT* cc = Ct + (size_t)col * ct_ld<DK, CT>() + a;
  const bool shared = (split & 31) != 0;
  if (packer) {
#pragma unroll
  for (int i0 = 0; i0 < HALF; i0 += CPR) {
    const uint4 raw = *(const uint4*)(cc + i0);
    const uint32_t pr[4] = {raw.x, raw.y, raw.z, raw.w};
    uint32_t wb[CPR / 4];
#pragma unroll
    for (int k = 0; k < CPR / 4; ++k) wb[k] = __builtin_amdgcn_readfirstlane(bw[i0 / 4 + k]);
#pragma unroll
    for (int u = 0; u < CPR; ++u) {
      const int b = (int)((wb[u / 4] >> (8 * (u % 4))) & 0xffu);
      const uint32_t field = __builtin_amdgcn_ubfe(pr[u / (4 / CB)], 8 * CB * (u % (4 / CB)), b);
      cur |= field << nb;
      nb += b;
      if (nb >= 32) {
        nb -= 32;
        if (first_pending) {
          first = cur;
          first_pending = false;
        } else {
          put(wi, cur);
        }
        ++wi;
        cur = field >> (b - nb);   // the nb bits that did not fit (0 if none)
      }
    }
  }
  // the lower half's last partial word goes to LDS when the upper half shares it
  if (half == 0 && nb > 0) {
    if (shared) tail[col] = cur;
    else put(wi, cur);
  }
  }
  __syncthreads();
  if (half == 1) {
    if (shared) {
      // first word of the upper half (complete, or still open if short)
      const uint32_t mine = first_pending ? cur : first;
      put(split >> 5, mine | tail[col]);
      if (!first_pending && nb > 0) put(wi, cur);
    } else if (nb > 0) {
      put(wi, cur);
    }
  }
}

// Write a record's metadata (header, widths, scales, stat codes).
// Rows [r0, r0 + ROWS) (r0 and ROWS even); the block of row 0 writes the header.
template <int DK, int ROWS = DK>
__device__ __forceinline__ void store_meta(uint8_t* rec, const Layout& L, unsigned ntok, const uint8_t* bits,
                           const uint16_t* scale16, const uint16_t* z, const uint16_t* r16,
                           int r0 = 0) {
  const int tid = threadIdx.x;
  if (r0 == 0 && tid < 4) ((unsigned*)rec)[tid] = tid == 0 ? ntok : 0u;
  if (tid < ROWS / 2) {
    const int q = r0 / 2 + tid;
    rec[L.w_off + q] = (uint8_t)((bits[2 * q] - 1) | ((bits[2 * q + 1] - 1) << 4));
  }
  if (tid < ROWS) {
    const int i = r0 + tid;
    ((uint16_t*)(rec + L.sc_off))[i] = scale16[i];
    ((uint16_t*)(rec + L.z_off))[i] = z[i];
    ((uint16_t*)(rec + L.r_off))[i] = r16[i];
  }
}

// Row loader of a row-major float32 state S[DK][DV]: segment sg of row i.
template <int DV>
__device__ __forceinline__ void load_dense(const float* S, int i, int sg, float (&x)[SEG]) {
  const float4* src = (const float4*)(S + (size_t)i * DV + sg * SEG);
#pragma unroll
  for (int q = 0; q < SEG / 4; ++q) {
    const float4 v = src[q];
    x[4 * q] = v.x;
    x[4 * q + 1] = v.y;
    x[4 * q + 2] = v.z;
    x[4 * q + 3] = v.w;
  }
}

// What the requantisation of a decode step needs besides its own tables when
// it rebuilds the state from the record: the record's decode metadata and the
// token's column vector w.
template <int DK, int DV, bool COMPACT>
struct RebuildLds {
  MetaSmem<DK> meta;
  float wv[DV];
};
template <int DK, int DV>
struct RebuildLds<DK, DV, false> {};

// LDS of the requantisation of one head.  With COMPACT the record's code
// words are staged column-major in the space of the code tile Ct (they are
// decoded before the first code is written).
template <int DK, int DV, bool COMPACT, typename CT>
struct RequantLds {
  RebuildLds<DK, DV, COMPACT> rb;
  __align__(16) CT Ct[DV * ct_ld<DK, CT>()];
  __align__(16) uint8_t nb[DK];
  uint8_t perm[DK];
  uint16_t sc16[DK], zz[DK], rr[DK];
  float phi[MAX_B + 1][N_FIT];
  OrderSmem<DK> os;
  uint32_t tail[DV];
};

// Threads of a requantisation block: 2 d_k, or one per (row, segment,
// candidate lane) of its dk / parts rows when that is more.
constexpr int requant_threads(int dk, int dv, int pairs, int parts = 1) {
  return 2 * dk > (dk / parts) * (dv / SEG) * pairs ? 2 * dk : (dk / parts) * (dv / SEG) * pairs;
}

// Quantise the state after the write-back interval with the allocated widths
// and pack it into the record in place (PAIRS: candidates per fit step, see
// fit_rows).  COMPACT (a decode step): the state is
// rebuilt row by row from the record and the token's vectors the stats pass
// left in the workspace, S_ij = fma(g_i, w_j, fl32(a_i x^_ij)) with x^ the
// record's dequantised value -- the same operations as the stats pass, so the
// same float32 state.  Otherwise the stats pass left the float32 state itself,
// and PARTS blocks may share the head: block `part` fits and packs rows
// [part DK / PARTS, (part + 1) DK / PARTS).  All threads of the block call it.
//
// ALLOC (prefill with the allocation weights in ws_c): the block first selects
// the widths of its scope unit itself (every block of the unit the same, by
// the same exact selection) and keeps those of its head, instead of reading
// the widths of a separate allocation launch.
template <int DK, int DV, bool COMPACT, typename CT, int PAIRS = 1, int PARTS = 1, bool ALLOC = false>
__device__ __forceinline__ void requant_head(const KParams& p, int bh, RequantLds<DK, DV, COMPACT, CT>& sm,
                                             int part = 0) {
  static_assert(!COMPACT || PARTS == 1, "the decode step rebuilds whole heads");
  constexpr int ROWS = DK / PARTS;
  const int r0 = part * ROWS;
  const Layout L = p.L;
  uint8_t* rec = (uint8_t*)slot_ptr(p.records, L.slot, bh);
  const int t = threadIdx.x;
  const unsigned ntok = *(const unsigned*)rec;
  // The float32 rows of this block's part (not the decode step: it rebuilds
  // its rows), when they fit in LDS: requested first, so that their latency
  // passes during the allocation and the width order, and read by the fit
  // from LDS.  Row r at sx[r SROW], segment g of it SEG + 4 floats further
  // per segment (the rows and segments of a wave's items fall in different
  // banks).
  constexpr int SROW = DV + 4 * (DV / SEG), NTH = requant_threads(DK, DV, PAIRS, PARTS);
  constexpr bool STAGE = !COMPACT && (size_t)ROWS * SROW * 4 <= 40 * 1024;
  constexpr int NV = STAGE ? ROWS * DV / 4 / NTH : 1;
  static_assert(!STAGE || (ROWS * DV / 4) % NTH == 0, "whole float4 per thread");
  typedef float v4f __attribute__((ext_vector_type(4)));   // held in registers, not copied through memory
  __shared__ __align__(16) float sx[STAGE ? ROWS * SROW : 4];
  v4f sv[NV];
  if constexpr (STAGE) {
    const v4f* S4 = (const v4f*)(p.ws_s32 + ((size_t)bh * DK + r0) * DV);
#pragma unroll
    for (int q = 0; q < NV; ++q) sv[q] = S4[t + q * NTH];
  }
  const uint32_t zr = t < DK ? p.ws_zr[(size_t)bh * DK + t] : 0u;
  if constexpr (ALLOC) {
    static_assert(!COMPACT && sizeof(AllocSmem) <= sizeof(sm.Ct), "allocator scratch in the code tile");
    // scope unit: the sequence (its heads' rows in order) or the head
    const int N = p.scope == 0 ? p.H * DK : DK;
    const int unit = p.scope == 0 ? bh / p.H : bh;
    const int row0 = p.scope == 0 ? (bh % p.H) * DK : 0;   // this head's first row in the unit
    constexpr int RPT = ALLOC_MAX_N / requant_threads(DK, DV, PAIRS, PARTS);
    block_allocate<RPT>([&](int n) { return p.ws_c[(size_t)unit * N + n]; }, N, p.need, p.bmin, p.bmax,
                        sm.nb, *(AllocSmem*)sm.Ct, row0, row0 + DK);
    __syncthreads();   // the head's widths are in nb; the tile is free again
  }
  if (t < DK) {
    if constexpr (!ALLOC) sm.nb[t] = (uint8_t)min(max((int)p.ws_bits[(size_t)bh * DK + t], 1), p.bmax);
    sm.zz[t] = (uint16_t)(zr & 0xffffu);
    sm.rr[t] = (uint16_t)(zr >> 16);
  }
  if constexpr (STAGE) {
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int e = 4 * (t + q * NTH), r = e / DV, c = e % DV;
      *(v4f*)&sx[r * SROW + c + 4 * (c / SEG)] = sv[q];
    }
  }
  for (int e = t; e < (MAX_B + 1) * N_FIT; e += blockDim.x)
    sm.phi[e / N_FIT][e % N_FIT] = p.phi[e / N_FIT][e % N_FIT];
  if constexpr (COMPACT) {
    // the staging needs DV (wc + 1) words, wc = ceil(d_k b_max / 32): 16-bit
    // tiles hold any b_max <= 16, byte tiles b_max <= 8 (the launcher's choice)
    static_assert((size_t)DV * (DK * (sizeof(CT) == 1 ? 8 : MAX_B) / 32 + 1) * 4 <= sizeof(sm.Ct),
                  "staging fits the code tile");
    const float* hv = p.ws_hv + (size_t)bh * (DV + 2 * DK);
    load_meta<DK, DV>(rec, L, p.bmax, sm.rb.meta);   // synchronises
    // the record's code words, column-major: word k of column j at
    // stg[j * STR + k], so a field that straddles two words is one pair; the
    // stride is the largest word count of any width bound the tile holds,
    // plus one (odd: the columns of a wave's lanes fall in distinct banks),
    // and a compile-time constant, so every read below is one immediate
    // offset from the lane's base address
    uint32_t* stg = (uint32_t*)sm.Ct;
    constexpr int STR = DK * (sizeof(CT) == 1 ? 8 : MAX_B) / 32 + 1;
    const int str = STR;
    const int nw = (sm.rb.meta.P[DK] + 31) >> 5;
    const uint4* src = (const uint4*)(rec + L.codes_off);
    for (int e = t; e < nw * (DV / 4); e += blockDim.x) {
      const int k = e / (DV / 4), c4 = e % (DV / 4);
      const uint4 v = src[(size_t)k * (DV / 4) + c4];
      stg[(4 * c4) * str + k] = v.x;
      stg[(4 * c4 + 1) * str + k] = v.y;
      stg[(4 * c4 + 2) * str + k] = v.z;
      stg[(4 * c4 + 3) * str + k] = v.w;
    }
    for (int e = t; e < DV; e += blockDim.x) sm.rb.wv[e] = hv[e];
    __syncthreads();
    width_order<DK>(sm.nb, sm.perm, sm.os, 0, DK, p.bmax);
    auto rebuild = [&](int i, int sg, float (&x)[SEG]) {
      const int P = sm.rb.meta.P[i];
      const int sh = P & 31, bo = sm.rb.meta.w[i];
      const uint4 d = sm.rb.meta.desc[i];
      const float mul = __builtin_bit_cast(float, d.z), add = __builtin_bit_cast(float, d.w);
      // x^ = fma(code, mul, add mul): the value of (code + add) mul for every
      // code (exact: add mul is 0 or mu, code mul is 0 or -2 mu for one-bit
      // rows), signed zeros aside, which no code or scale below depends on
      const float addm = add * mul;
      const float ai = hv[DV + i], gi = hv[DV + DK + i];
      const uint32_t* cw = stg + (size_t)(sg * SEG) * str + (P >> 5);
#pragma unroll
      for (int j = 0; j < SEG; ++j) {
        const uint32_t lo = cw[j * str], hi = cw[j * str + 1];
        const uint32_t f = __builtin_amdgcn_alignbit(hi, lo, (uint32_t)sh);
        const int code = __builtin_amdgcn_sbfe((int)f, 0, bo);   // signed field
        const float xh = __builtin_fmaf((float)code, mul, addm);
        x[j] = __builtin_fmaf(gi, sm.rb.wv[sg * SEG + j], ai * xh);
      }
    };
    fit_rows<DK, DV, true>(rebuild, sm.nb, sm.perm, sm.phi, sm.Ct, sm.sc16, p.diag_fit);
  } else {
    __syncthreads();
    width_order<DK>(sm.nb, sm.perm, sm.os, r0, r0 + ROWS, p.bmax);
    const float* S = p.ws_s32 + (size_t)bh * DK * DV;
    auto staged = [&](int i, int sg, float (&x)[SEG]) {
      const int li = min(max(i - r0, 0), ROWS - 1);
      const float4* src = (const float4*)&sx[li * SROW + sg * (SEG + 4)];
#pragma unroll
      for (int q = 0; q < SEG / 4; ++q) {
        const float4 v = src[q];
        x[4 * q] = v.x;
        x[4 * q + 1] = v.y;
        x[4 * q + 2] = v.z;
        x[4 * q + 3] = v.w;
      }
    };
    auto dense = [&](int i, int sg, float (&x)[SEG]) { load_dense<DV>(S, i, sg, x); };
    if constexpr (STAGE)
      fit_rows<DK, DV, false, PAIRS, ROWS>(staged, sm.nb, sm.perm, sm.phi, sm.Ct, sm.sc16, p.diag_fit);
    else
      fit_rows<DK, DV, false, PAIRS, ROWS>(dense, sm.nb, sm.perm, sm.phi, sm.Ct, sm.sc16, p.diag_fit);
  }
  __syncthreads();
  pack_cols<DK, DV, ROWS>(sm.Ct, sm.nb, sm.os.P, (uint32_t*)(rec + L.codes_off), sm.tail, r0);
  store_meta<DK, ROWS>(rec, L, ntok + (unsigned)p.ntk, sm.nb, sm.sc16, sm.zz, sm.rr, r0);
}

// Code tile element: bytes when widths fit (b_max <= 8), else 16 bits.
template <bool C8>
using CodeTile = typename std::conditional<C8, int8_t, int16_t>::type;

}  // namespace kda
