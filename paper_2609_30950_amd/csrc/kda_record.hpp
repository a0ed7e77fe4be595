// Record access shared by the kernels: slot addressing, the per-row
// metadata of a stored record and its decode descriptors, and token-input
// loads (bf16 bit patterns or float32).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kda_device.hpp"

namespace kda {

// Columns of one prefill column slice (one block per slice and head).
constexpr int SLICE = 64;

// Block of a per-slice kernel: (head, 64-column slice).  Workgroups are
// dealt to the eight XCDs in turn, so the slices of one head are placed 8
// block indices apart: they run on one XCD, and what they both read (the
// head's metadata, token inputs, chunk records) comes from that XCD's L2
// after the first read.  Heads past the last multiple of 8 map in order.
__device__ __forceinline__ void slice_block(int nbh, int nsl, int& bh, int& sl) {
  constexpr int XCD = 8;
  const int id = blockIdx.x, full = (nbh / XCD) * XCD * nsl;
  if (id < full) {
    sl = (id / XCD) % nsl;
    bh = id % XCD + XCD * (id / (XCD * nsl));
  } else {
    bh = (nbh / XCD) * XCD + (id - full) / nsl;
    sl = (id - full) % nsl;
  }
}

__device__ __forceinline__ const uint8_t* slot_ptr(const void* recs, long long slot, int bh) {
  return (const uint8_t*)recs + slot * (long long)bh;
}

template <int DK>
struct MetaSmem {
  // per-row decode descriptor, read by whole waves as one broadcast:
  // {first word index * d_v, bit shift | width << 8, mul, add} (see unpack_cols)
  uint4 desc[DK];
  uint8_t w[DK];      // widths of the stored record
  int P[DK + 1];      // prefix sums of widths (row bit offsets)
  uint16_t sc[DK];    // stored scales (FP16 bits)
  uint16_t z[DK];     // stored rate codes
  uint16_t r16[DK];   // stored erase rates
  unsigned ntok;
};

// A record's stored metadata as one thread reads it (thread t < d_k: row t's
// scale and codes; t < d_k / 2: the byte of rows 2t and 2t + 1; thread 0: the
// token count), held in registers until meta_form writes it out.
struct MetaFetch {
  uint32_t wb, sc, z, r, ntok;
};

template <int DK>
__device__ __forceinline__ MetaFetch meta_fetch(const uint8_t* rec, const Layout& L) {
  const int tid = threadIdx.x;
  MetaFetch f{0u, 0u, 0u, 0u, 0u};
  if (tid < DK / 2) f.wb = rec[L.w_off + tid];
  if (tid < DK) {
    f.sc = ((const uint16_t*)(rec + L.sc_off))[tid];
    f.z = ((const uint16_t*)(rec + L.z_off))[tid];
    f.r = ((const uint16_t*)(rec + L.r_off))[tid];
  }
  if (tid == 0) f.ntok = *(const unsigned*)rec;
  return f;
}

// Widths/scales/stat codes of a record and its row offsets and decode
// descriptors, from what meta_fetch read.  Widths above b_max (never written
// by this library) are clamped so that a damaged record cannot address code
// words outside its slot.
template <int DK, int DV>
__device__ __forceinline__ void meta_form(const MetaFetch& f, int bmax, MetaSmem<DK>& m) {
  const int tid = threadIdx.x;
  if (tid < DK / 2) {
    m.w[2 * tid] = (uint8_t)min((int)(f.wb & 15u) + 1, bmax);
    m.w[2 * tid + 1] = (uint8_t)min((int)(f.wb >> 4) + 1, bmax);
  }
  if (tid < DK) {
    m.sc[tid] = (uint16_t)f.sc;
    m.z[tid] = (uint16_t)f.z;
    m.r16[tid] = (uint16_t)f.r;
  }
  if (tid == 0) m.ntok = f.ntok;
  __syncthreads();
  if (tid < WAVE) {
    constexpr int PER = (DK + WAVE - 1) / WAVE;
    int loc[PER], sum = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int i = tid * PER + q;
      loc[q] = i < DK ? m.w[i] : 0;
      sum += loc[q];
    }
    const int incl = wave_incl_scan(sum);
    int run = incl - sum;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int i = tid * PER + q;
      if (i < DK) {
        m.P[i] = run;
        // x^ = (code + add) mul: (Delta, 0) for b >= 2, (2 mu, 1/2) for one bit
        const int b = loc[q];
        const float sc = f16_to_f32(m.sc[i]);
        const float mul = b == 1 ? 2.0f * sc : sc;
        const float add = b == 1 ? 0.5f : 0.0f;
        m.desc[i] = make_uint4((uint32_t)((run >> 5) * DV), (uint32_t)((run & 31) | (b << 8)),
                               __builtin_bit_cast(uint32_t, mul), __builtin_bit_cast(uint32_t, add));
      }
      run += loc[q];
    }
    if (tid == WAVE - 1) m.P[DK] = incl;
  }
  __syncthreads();
}

// Load a record's metadata and form the row offsets (both steps at once).
template <int DK, int DV>
__device__ __forceinline__ void load_meta(const uint8_t* rec, const Layout& L, int bmax, MetaSmem<DK>& m) {
  meta_form<DK, DV>(meta_fetch<DK>(rec, L), bmax, m);
}

template <bool BF16>
__device__ __forceinline__ float in_f32(const void* base, size_t idx) {
  if constexpr (BF16) return __builtin_bit_cast(float, (uint32_t)((const uint16_t*)base)[idx] << 16);
  return ((const float*)base)[idx];
}

}  // namespace kda
