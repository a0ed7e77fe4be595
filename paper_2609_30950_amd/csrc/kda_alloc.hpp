// Exact integer bit allocation for one scope unit, executed by one block.
//
// Minimises sum_i c_i 2^(-2 b_i) over b_i in [b_min, b_max] with a fixed
// total (Sec. 3, eq. alloc, rounded/clipped/adjusted to the budget).  Every
// row owns slots l = b_min+1..b_max worth c_i 4^(-l); the `need` largest slots
// are granted, ties to the lower row index (then lower l).
//
// Slot keys are compared exactly as (E_i - 2 l, M_i) with c_i = M_i 2^E_i,
// M_i in [0.5, 1) (frexp).  The selection runs in exact stages:
//  1. bucket E - 2l: a histogram of the row exponents (LDS atomics) gives the
//     slot count of every bucket; the boundary bucket beta* is the highest one
//     at which the running count from the top reaches `need`;
//  2. rows owning a slot in beta* (at most one slot per row) are narrowed by
//     radix passes over the 52 fraction bits (256-bin LDS histograms), each
//     keeping the digit bin that contains the boundary, until at most one
//     wave of candidates remains;
//  3. those are ranked by (fraction desc, row asc), one ballot per
//     candidate, and the first ones granted.
// Rows with c_i = 0 own slots below every positive one, granted in row order.
#pragma once

#include "kda_device.hpp"
#include "kda_kernels.hpp"

namespace kda {

constexpr int ALLOC_MAX_N = 4096;     // rows per scope unit
constexpr int ALLOC_MAX_T = 1024;     // threads per block
constexpr int E_ZERO = -100000;       // exponent sentinel of c = 0
constexpr int EBINS = 2304;           // exponent histogram range (frexp: [-1073, 1024])
constexpr int EOFF = 1100;

struct AllocSmem {
  int hist_e[EBINS];
  int hist_d[2][256];   // digit histograms of consecutive radix passes
  int red[48];
  int cand_n;
  int npos, emin, emax;
  int sel_beta, sel_digit, sel_rem, sel_live;
  unsigned long long cand_key[WAVE];
  int cand_row[WAVE];
  unsigned char extra[ALLOC_MAX_N];
};

__device__ __forceinline__ int slots_ge(int E, int beta, int bmin, int L) {
  if (E == E_ZERO) return 0;
  const int lmax = (E - beta) >> 1;  // floor division
  const int c = lmax - bmin;
  return c < 0 ? 0 : (c > L ? L : c);
}

// Block-wide exclusive scan of one int per thread (row order = thread order).
__device__ __forceinline__ int block_excl_scan(int v, int* scratch, int* total) {
  const int w = threadIdx.x / WAVE, nw = (blockDim.x + WAVE - 1) / WAVE;
  const int incl = wave_incl_scan(v);
  __syncthreads();
  if (lane_id() == WAVE - 1) scratch[w] = incl;
  __syncthreads();
  int off = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < w) off += scratch[i];
    tot += scratch[i];
  }
  *total = tot;
  return off + incl - v;
}

// 52 fraction bits of the frexp mantissa of c > 0 (c = (1 + F 2^-52) 2^(E-1)).
__device__ __forceinline__ unsigned long long frac_bits(double c) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(c);
  if ((u >> 52) != 0ull) return u & ((1ull << 52) - 1ull);   // normal: the stored fraction
  int e;
  const double m = frexp(c, &e);
  return (unsigned long long)ldexp(m, 53) - (1ull << 52);
}

// c_at(n): weight of row n (any address space); out[n - lo]: the widths of
// rows lo <= n < hi (the rest are not written).  RPT: rows per thread, at least
// ceil(N / blockDim.x).
template <int RPT, typename Load>
__device__ __forceinline__ void block_allocate(Load c_at, int N, int need, int bmin, int bmax, uint8_t* out,
                               AllocSmem& sm, int lo = 0, int hi = 0x7fffffff) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = lane_id();
  const int L = bmax - bmin;
  // rows n = tid + k * nt, k < RPT, their weights held in registers (read
  // once: the radix passes and the ranking use them again)
  static_assert(RPT <= 32, "candidate mask");
  int E[RPT];
  double Cv[RPT];
  // weights first: their load latency overlaps the clearing of the histograms
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int n = tid + k * nt;
    Cv[k] = n < N ? c_at(n) : 0.0;
  }
  for (int e = tid; e < EBINS; e += nt) sm.hist_e[e] = 0;
  for (int e = tid; e < 2 * 256; e += nt) sm.hist_d[e >> 8][e & 255] = 0;
  for (int n = tid; n < N; n += nt) sm.extra[n] = 0;
  if (tid == 0) {
    sm.cand_n = 0;
    sm.npos = 0;
    sm.emin = 0x7fffffff;
    sm.emax = -0x7fffffff;
  }
  int npos = 0, emin = 0x7fffffff, emax = -0x7fffffff;
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    E[k] = E_ZERO;
    {
      const double cv = Cv[k];
      if (cv > 0.0) {
        int ei;
        frexp(cv, &ei);
        E[k] = ei;
        ++npos;
        emin = min(emin, ei);
        emax = max(emax, ei);
      }
    }
  }
  __syncthreads();
  // histogram of exponents (one LDS atomic per row: the exponents of a
  // wave's rows are too varied for per-value aggregation to pay); count and
  // exponent range reduced per wave, one LDS atomic each
#pragma unroll
  for (int k = 0; k < RPT; ++k)
    if (E[k] != E_ZERO) atomicAdd(&sm.hist_e[E[k] + EOFF], 1);
  npos = wave_reduce_i(npos, [](int a, int b) { return a + b; });
  emin = wave_reduce_i(emin, [](int a, int b) { return a < b ? a : b; });
  emax = wave_reduce_i(emax, [](int a, int b) { return a > b ? a : b; });
  if (lane == 0) {
    atomicAdd(&sm.npos, npos);
    atomicMin(&sm.emin, emin);
    atomicMax(&sm.emax, emax);
  }
  __syncthreads();
  npos = sm.npos;
  emin = sm.emin;
  emax = sm.emax;
  const long long ptot = (long long)npos * L;

  if (need <= 0) {
    for (int n = tid; n < N; n += nt)
      if (n >= lo && n < hi) out[n - lo] = (uint8_t)bmin;
    return;
  }
  if (ptot <= need) {
    // every positive slot, then zero rows in row order
    const long long rem0 = need - ptot;
    int carry = 0;
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int n = tid + k * nt;
      const int isz = (n < N && E[k] == E_ZERO) ? 1 : 0;
      int tot;
      const int z = carry + block_excl_scan(isz, sm.red, &tot);
      if (n < N) {
        int b;
        if (!isz) {
          b = bmax;
        } else {
          long long g = rem0 - (long long)L * z;
          g = g < 0 ? 0 : (g > L ? L : g);
          b = bmin + (int)g;
        }
        if (n >= lo && n < hi) out[n - lo] = (uint8_t)b;
      }
      carry += tot;
      __syncthreads();
    }
    return;
  }

  // stage 1: boundary bucket from the exponent histogram.  Bucket bb holds
  // sum_l hist[bb + 2l] slots; wave 0 examines 64 buckets at a time from the
  // top and finds the first at which the running count reaches `need`.
  if (tid < WAVE) {
    const int top = emax - 2 * (bmin + 1);
    const int bot = emin - 2 * bmax;
    int run = 0;
    for (int b0 = top; b0 >= bot; b0 -= WAVE) {
      const int bb = b0 - lane;
      int cnt = 0;
      if (bb >= bot)
        for (int l = bmin + 1; l <= bmax; ++l) {
          const int e = bb + 2 * l + EOFF;
          if (e >= 0 && e < EBINS) cnt += sm.hist_e[e];
        }
      // inclusive prefix over lanes (lane order = descending bucket)
      const int incl = wave_incl_scan(cnt);
      const unsigned long long hit = __ballot(run + incl >= need);
      if (hit) {
        const int f = __ffsll((long long)hit) - 1;
        if (lane == f) {
          sm.sel_beta = bb;
          sm.sel_rem = (int)(need - (run + incl - cnt));
          sm.sel_live = cnt;   // rows with a slot in bucket bb: the candidates
        }
        break;
      }
      run += __builtin_amdgcn_readlane(incl, WAVE - 1);
    }
  }
  __syncthreads();
  const int beta = sm.sel_beta;
  int rem = sm.sel_rem;
  int live = sm.sel_live;

  // stage 2: radix narrowing of the candidates of bucket beta (bit k of cand:
  // row tid + k nt is a candidate)
  unsigned cand = 0u;
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    if (E[k] != E_ZERO && ((E[k] - beta) & 1) == 0) {
      const int l = (E[k] - beta) >> 1;
      if (l >= bmin + 1 && l <= bmax) cand |= 1u << k;
    }
  }
  // each pass: histogram of the candidates' next digit, the digit bin that
  // holds the boundary (wave 0; the other waves clear the next pass's
  // histogram meanwhile), then candidates above it are granted and below it
  // dropped; the bin's count is the next pass's number of candidates
  bool many = true;
  for (int pass = 0; pass < 7; ++pass) {
    if (live <= WAVE) { many = false; break; }
    const int shift = pass < 6 ? 44 - 8 * pass : 0;
    const unsigned long long dmask = pass < 6 ? 255ull : 15ull;
    int* hd = sm.hist_d[pass & 1];
#pragma unroll
    for (int k = 0; k < RPT; ++k)
      if ((cand >> k) & 1u) atomicAdd(&hd[(frac_bits(Cv[k]) >> shift) & dmask], 1);
    __syncthreads();
    if (tid < WAVE) {
      // lane j covers bins 4j+3..4j of the descending order dmask..0
      int h[4], tot = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = (int)dmask - (4 * lane + u);
        h[u] = d >= 0 ? hd[d] : 0;
        tot += h[u];
      }
      const int incl = wave_incl_scan(tot);
      const unsigned long long hit = __ballot(incl >= rem);
      const int f = __ffsll((long long)hit) - 1;
      if (lane == f) {
        int run = incl - tot;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (run + h[u] >= rem) {
            sm.sel_digit = (int)dmask - (4 * lane + u);
            sm.sel_rem = rem - run;
            sm.sel_live = h[u];
            break;
          }
          run += h[u];
        }
      }
      if (nt == WAVE)
        for (int e = lane; e < 256; e += WAVE) sm.hist_d[(pass + 1) & 1][e] = 0;
    } else {
      for (int e = tid - WAVE; e < 256; e += nt - WAVE) sm.hist_d[(pass + 1) & 1][e] = 0;
    }
    __syncthreads();
    const unsigned long long dg = (unsigned long long)sm.sel_digit;
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      if (!((cand >> k) & 1u)) continue;
      const unsigned long long d = (frac_bits(Cv[k]) >> shift) & dmask;
      if (d > dg) {
        sm.extra[tid + k * nt] = 1;   // above the boundary digit: granted
        cand &= ~(1u << k);
      } else if (d < dg) {
        cand &= ~(1u << k);
      }
    }
    rem = sm.sel_rem;
    live = sm.sel_live;
  }
  if (many) {
    // more than a wave of candidates with identical keys: lowest rows first
    int carry = 0;
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      int tot;
      const int ck = (cand >> k) & 1u;
      const int z = carry + block_excl_scan(ck, sm.red, &tot);
      if (ck && z < rem) sm.extra[tid + k * nt] = 1;
      carry += tot;
      __syncthreads();
    }
    cand = 0u;
  }
  // stage 3: at most one wave of candidates left: rank them
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    if (!((cand >> k) & 1u)) continue;
    const int pos = atomicAdd(&sm.cand_n, 1);
    sm.cand_key[pos] = frac_bits(Cv[k]);
    sm.cand_row[pos] = tid + k * nt;
  }
  __syncthreads();
  {
    // the candidates' ranks by (fraction desc, row asc), every wave taking
    // some of them: candidate i's rank is the number of lanes j whose
    // candidate comes first (one ballot per candidate)
    const int nc = sm.cand_n, nw = nt / WAVE, wv = tid / WAVE;
    const unsigned long long kj = lane < nc ? sm.cand_key[lane] : 0ull;
    const int rj = lane < nc ? sm.cand_row[lane] : 0;
    for (int i = wv; i < nc; i += nw) {
      const unsigned long long ki = sm.cand_key[i];
      const int ri = sm.cand_row[i];
      const bool first = lane < nc && (kj > ki || (kj == ki && rj < ri));
      const int rank = __popcll(__ballot(first));
      if (lane == 0 && rank < rem) sm.extra[ri] = 1;
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int n = tid + k * nt;
    if (n < N && n >= lo && n < hi) out[n - lo] = (uint8_t)(bmin + slots_ge(E[k], beta + 1, bmin, L) + sm.extra[n]);
  }
}

// Row statistics of one write-back for one head (threads t < DK own row t).
template <int DK>
struct StatSmem {
  float R[DK];     // first member: 16-byte aligned with the struct
  double gam[DK];
  double rms[DK];
  double c[DK];
};

// Sum of squares of the float32 values x[r0..r1) in float64, in order; with
// 16-byte aligned bounds the reads are issued four values at a time ahead of
// the sequential sum.
__device__ __forceinline__ double run_sumsq(const float* x, int r0, int r1) {
  double acc = 0.0;
  int j = r0;
  if (((r0 | r1) & 3) == 0) {
    const float4* x4 = (const float4*)(x + r0);
#pragma unroll 4
    for (; j < r1; j += 4) {
      const float4 v = x4[(j - r0) >> 2];
      acc = acc + (double)v.x * (double)v.x;
      acc = acc + (double)v.y * (double)v.y;
      acc = acc + (double)v.z * (double)v.z;
      acc = acc + (double)v.w * (double)v.w;
    }
  }
  for (; j < r1; ++j) acc = acc + (double)x[j] * (double)x[j];
  return acc;
}

// Weights c = Gamma R~^2 from the row ranges st.R (group RMS in float64: the
// squares summed in runs of RMS_RUN rows, each run in row order, the run
// sums in order).  The caller has synchronised after writing st.R.
template <int DK>
__device__ __forceinline__ void row_weights(const KParams& p, int bh, StatSmem<DK>& st, int t) {
  const int G = p.G, runs = (G + RMS_RUN - 1) / RMS_RUN;
  if (t < (DK / G) * runs) {
    const int g = t / runs, r0 = g * G + (t % runs) * RMS_RUN;
    st.c[t] = run_sumsq(st.R, r0, min(r0 + RMS_RUN, (g + 1) * G));   // run sums, in the
    // space of the weights until those are formed
  }
  __syncthreads();
  if (t < DK / G) {
    double acc = 0.0;
    for (int k = 0; k < runs; ++k) acc = acc + st.c[t * runs + k];
    st.rms[t] = sqrt(acc / (double)G);
  }
  __syncthreads();
  if (t < DK) {
    const double c = mode_key(p.weight_mode, st.gam[t], st.R[t], st.rms[t / p.G]);
    st.c[t] = c;
    p.ws_c[(size_t)bh * DK + t] = c;
  }
  __syncthreads();
}

}  // namespace kda
