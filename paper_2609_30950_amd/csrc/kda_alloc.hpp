// Exact integer bit allocation for one scope unit, executed by one block.
//
// Minimises sum_i c_i 2^(-2 b_i) over b_i in [b_min, b_max] with a fixed
// total (Sec. 3, eq. alloc, rounded/clipped/adjusted to the budget).  Every
// row owns slots l = b_min+1..b_max worth c_i 4^(-l); the `need` largest slots
// are granted, ties to the lower row index (then lower l).
//
// Slot keys are compared exactly as (E_i - 2 l, M_i) with c_i = M_i 2^E_i,
// M_i in [0.5, 1) (frexp).  The search runs in two exact stages:
//  1. bisection on the integer bucket E - 2 l: the largest bucket beta* such
//     that at least `need` slots lie in buckets >= beta*;
//  2. the rows owning a slot in bucket beta* (at most one slot per row) are
//     sorted by (M desc, row asc) with an LDS bitonic sort and the first
//     `need - (slots above beta*)` of them are granted that slot.
// Rows with c_i = 0 own slots below every positive one, granted in row order.
#pragma once

#include "kda_device.hpp"

namespace kda {

constexpr int ALLOC_MAX_N = 4096;  // rows per scope unit (12-bit row field)
constexpr short E_ZERO = -32768;   // exponent sentinel of c = 0

struct AllocSmem {
  short E[ALLOC_MAX_N];
  unsigned long long keys[ALLOC_MAX_N];
  unsigned char extra[ALLOC_MAX_N];
  int red_i[32];
  long long red_l[32];
  int ncand;
};

__device__ inline int slots_ge(int E, int beta, int bmin, int L) {
  if (E == E_ZERO) return 0;
  int lmax = (E - beta) >> 1;  // floor division
  int c = lmax - bmin;
  return c < 0 ? 0 : (c > L ? L : c);
}

// Block-wide exclusive scan of one int per thread (row order = thread order).
__device__ inline int block_excl_scan(int v, int* scratch, int* total) {
  const int w = threadIdx.x / WAVE, nw = (blockDim.x + WAVE - 1) / WAVE;
  int incl = wave_incl_scan(v);
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

// c: N weights (any address space readable by the block); out: N widths.
template <typename Load>
__device__ void block_allocate(Load c_at, int N, int need, int bmin, int bmax,
                               uint8_t* out, AllocSmem& sm) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int L = bmax - bmin;
  int emin = 0x7fffffff, emax = -0x7fffffff, npos = 0;
  for (int n = tid; n < N; n += nt) {
    const double cv = c_at(n);
    short e = E_ZERO;
    if (cv > 0.0) {
      int ei;
      (void)frexp(cv, &ei);
      e = (short)ei;
      emin = min(emin, ei);
      emax = max(emax, ei);
      ++npos;
    }
    sm.E[n] = e;
    sm.extra[n] = 0;
  }
  emin = block_reduce(emin, sm.red_i, [](int a, int b) { return a < b ? a : b; });
  emax = block_reduce(emax, sm.red_i, [](int a, int b) { return a > b ? a : b; });
  npos = block_reduce(npos, sm.red_i, [](int a, int b) { return a + b; });
  __syncthreads();
  const long long ptot = (long long)npos * L;

  if (need <= 0) {
    for (int n = tid; n < N; n += nt) out[n] = (uint8_t)bmin;
    return;
  }
  if (ptot <= need) {
    // every positive slot, then zero rows in row order
    const long long rem0 = need - ptot;
    int carry = 0;
    for (int base = 0; base < N; base += nt) {
      const int n = base + tid;
      const int isz = (n < N && sm.E[n] == E_ZERO) ? 1 : 0;
      int tot;
      const int z = carry + block_excl_scan(isz, sm.red_i, &tot);
      if (n < N) {
        int b;
        if (!isz) {
          b = bmax;
        } else {
          long long g = rem0 - (long long)L * z;
          g = g < 0 ? 0 : (g > L ? L : g);
          b = bmin + (int)g;
        }
        out[n] = (uint8_t)b;
      }
      carry += tot;
      __syncthreads();
    }
    return;
  }

  // stage 1: bucket bisection
  int lo = emin - 2 * bmax, hi = emax - 2 * (bmin + 1);
  while (lo < hi) {
    const int mid = lo + ((hi - lo + 1) >> 1);
    long long cnt = 0;
    for (int n = tid; n < N; n += nt) cnt += slots_ge(sm.E[n], mid, bmin, L);
    cnt = block_reduce(cnt, sm.red_l, [](long long a, long long b) { return a + b; });
    if (cnt >= need) lo = mid; else hi = mid - 1;
  }
  const int beta = lo;
  long long ngt = 0;
  for (int n = tid; n < N; n += nt) ngt += slots_ge(sm.E[n], beta + 1, bmin, L);
  ngt = block_reduce(ngt, sm.red_l, [](long long a, long long b) { return a + b; });
  const long long rem = need - ngt;  // >= 1 slots taken inside bucket beta

  // stage 2: candidates of bucket beta
  if (tid == 0) sm.ncand = 0;
  __syncthreads();
  for (int base = 0; base < N; base += nt) {
    const int n = base + tid;
    bool cand = false;
    unsigned long long key = 0;
    if (n < N) {
      const int e = sm.E[n];
      if (e != E_ZERO && ((e - beta) & 1) == 0) {
        const int l = (e - beta) >> 1;
        if (l >= bmin + 1 && l <= bmax) {
          int ei;
          const double m = frexp(c_at(n), &ei);           // [0.5, 1)
          const unsigned long long m53 = (unsigned long long)ldexp(m, 53);
          key = ((m53 - (1ull << 52)) << 12) | (unsigned long long)(ALLOC_MAX_N - 1 - n);
          cand = true;
        }
      }
    }
    const unsigned long long mask = __ballot(cand);
    int wbase = 0;
    if (lane_id() == 0 && mask) wbase = atomicAdd(&sm.ncand, __popcll(mask));
    wbase = __shfl(wbase, 0, WAVE);
    if (cand) {
      const int pos = wbase + __popcll(mask & ((1ull << lane_id()) - 1ull));
      sm.keys[pos] = key;
    }
  }
  __syncthreads();
  const int nc = sm.ncand;
  if (rem >= nc) {
    for (int p = tid; p < nc; p += nt)
      sm.extra[ALLOC_MAX_N - 1 - (int)(sm.keys[p] & 4095ull)] = 1;
  } else {
    int p2 = 1;
    while (p2 < nc) p2 <<= 1;
    for (int p = nc + tid; p < p2; p += nt) sm.keys[p] = 0ull;
    __syncthreads();
    for (int k = 2; k <= p2; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int t = tid; t < (p2 >> 1); t += nt) {
          const int i = (t / j) * 2 * j + (t % j);
          const int l = i + j;
          const bool up = (i & k) == 0;
          const unsigned long long a = sm.keys[i], b = sm.keys[l];
          if ((a < b) == up) { sm.keys[i] = b; sm.keys[l] = a; }
        }
        __syncthreads();
      }
    }
    for (int p = tid; p < (int)rem; p += nt)
      sm.extra[ALLOC_MAX_N - 1 - (int)(sm.keys[p] & 4095ull)] = 1;
  }
  __syncthreads();
  for (int n = tid; n < N; n += nt)
    out[n] = (uint8_t)(bmin + slots_ge(sm.E[n], beta + 1, bmin, L) + sm.extra[n]);
}

}  // namespace kda
