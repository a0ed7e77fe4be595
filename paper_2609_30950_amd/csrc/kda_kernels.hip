// HIP kernels of libkda for gfx950 (MI355X), wave64.
//
// One workgroup per (sequence, head).  Two thread layouts are used:
//  * column layout (recurrence, unpack, pack): wave w owns rows
//    [32w, 32w + 32) and lane l owns columns l + 64c, c < d_v/64.  The row
//    contractions u = S'^T k and o = S^T q are then sequential fma chains in
//    registers (one 32-row block per wave) plus a halving combine of the
//    per-wave partials through LDS; every row's width, offset and scale is
//    wave-uniform, so bit fields are extracted with uniform shifts.
//  * row layout (fit): after an LDS transpose, thread t owns one 64-column
//    segment of one row; the clip-factor fit needs no cross-lane traffic
//    except the combine of the d_v/64 segment errors of a row.
//
// Decode (C = 1) runs three kernels: stats (recurrence, outputs, row ranges,
// EMA rates, weights), alloc (layer budget per sequence; skipped for the
// per-head scope, which allocates inside stats) and requant (recompute the
// recurrence from the record, fit, quantise, pack in place).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kda_alloc.hpp"
#include "kda_device.hpp"
#include "kda_kernels.hpp"
#include "kda_profile.hpp"
#include "kda_record.hpp"
#include "kda_recur.hpp"
#include "kda_requant.hpp"

namespace kda {

// ------------------------------------------------------------ helpers ---

// Copy the meaningful code words of a record (ceil(sum b / 32) words per
// column) into LDS with coalesced 16-byte loads.  All threads must call.
template <int DV, bool SYNC = true>
__device__ __forceinline__ void stage_words(const uint8_t* rec, const Layout& L, int total_bits, uint32_t* lds) {
  const int nw = (total_bits + 31) >> 5;
  const int n4 = nw * DV / 4;
  const uint4* src = (const uint4*)(rec + L.codes_off);
  uint4* dst = (uint4*)lds;
  for (int e = threadIdx.x; e < n4; e += blockDim.x) dst[e] = src[e];
  if constexpr (SYNC) __syncthreads();
}

// Decode staged code words into column-layout registers X[r][c] (row
// 32w + r, column lane + 64c): x^ = fl32(code * Delta), or +-mu for one-bit
// rows.  Each row's descriptor is one LDS broadcast read; its word index,
// shift and width are wave-uniform (scalar registers).  One expression covers
// every width: the field is sign-extended, then x^ = (code + add) mul with
// (mul, add) = (Delta, 0) for b >= 2, which is fl32(code Delta), and
// (2 mu, 1/2) for one-bit rows (code 0 or -1), which gives mu or -mu exactly,
// signed zeros included.
template <int DK, int DV>
__device__ __forceinline__ void unpack_cols(const uint32_t* words, const MetaSmem<DK>& m,
                            float (&X)[ROW_BLOCK][DV / WAVE]) {
  constexpr int CPL = DV / WAVE;
  const int w = threadIdx.x / WAVE, lane = lane_id();
#pragma unroll
  for (int r = 0; r < ROW_BLOCK; ++r) {
    const uint4 d = m.desc[w * ROW_BLOCK + r];
    const int base = __builtin_amdgcn_readfirstlane((int)d.x);
    const int shb = __builtin_amdgcn_readfirstlane((int)d.y);
    const int sh = shb & 31, b = shb >> 8;
    const float mul = __builtin_bit_cast(float, d.z), add = __builtin_bit_cast(float, d.w);
    const uint32_t* wr = words + base;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int col = lane + WAVE * c;
      const uint32_t lo = wr[col];
      const uint32_t hi = wr[DV + col];   // staged; masked off unless straddling
      const uint32_t f = __builtin_amdgcn_alignbit(hi, lo, (uint32_t)sh);
      const int code = __builtin_amdgcn_sbfe((int)f, 0, b);
      // add is +0 for widths >= 2: code + 0 is code exactly (no select per row)
      X[r][c] = ((float)code + add) * mul;
    }
    // finish row r before the reads of later rows are issued: the compiler
    // would otherwise keep every row's descriptor and words live at once
    if (r % 4 == 3) {
#pragma unroll
      for (int q = r - 3; q <= r; ++q)
#pragma unroll
        for (int c = 0; c < CPL; ++c) asm volatile("" : "+v"(X[q][c])::"memory");
    }
  }
}

// Row absolute maxima of column-layout registers into R[DK].  Reduce-scatter
// over the 64 lanes: each step halves the number of row values per lane by
// pairing lanes that differ in one bit (permlane32/16 swaps for bits 5 and 4,
// DPP rotates within 16-lane rows for bits 3 and 2, quad permutes for bits 1
// and 0).  Afterwards lanes 2r and 2r+1 of wave w hold row 32w + r.
template <int CTRL>
__device__ __forceinline__ float fmax_dpp(float v) { return fmaxf(v, dpp_f<CTRL>(v)); }

__device__ __forceinline__ float swap_max32(float a, float b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, a), __builtin_bit_cast(int, b),
                                                  false, false);
  return fmaxf(__builtin_bit_cast(float, (int)r[0]), __builtin_bit_cast(float, (int)r[1]));
}

__device__ __forceinline__ float swap_max16(float a, float b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, a), __builtin_bit_cast(int, b),
                                                  false, false);
  return fmaxf(__builtin_bit_cast(float, (int)r[0]), __builtin_bit_cast(float, (int)r[1]));
}

template <int DK, int DV>
__device__ __forceinline__ void row_max(const float (&X)[ROW_BLOCK][DV / WAVE], float* R) {
  constexpr int CPL = DV / WAVE;
  const int w = threadIdx.x / WAVE, lane = lane_id();
  float v[ROW_BLOCK];
#pragma unroll
  for (int r = 0; r < ROW_BLOCK; ++r) {
    float mx = fabsf(X[r][0]);
#pragma unroll
    for (int c = 1; c < CPL; ++c) mx = fmaxf(mx, fabsf(X[r][c]));
    v[r] = mx;
  }
  // lane bit 5: rows r and r + 16
#pragma unroll
  for (int r = 0; r < 16; ++r) v[r] = swap_max32(v[r], v[r + 16]);
  // lane bit 4: rows r and r + 8
#pragma unroll
  for (int r = 0; r < 8; ++r) v[r] = swap_max16(v[r], v[r + 8]);
  const bool b3 = (lane >> 3) & 1, b2 = (lane >> 2) & 1, b1 = (lane >> 1) & 1;
  // lane bit 3 (rotate by 8 inside 16-lane rows is its own inverse)
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float x0 = fmax_dpp<0x128>(v[r]), x1 = fmax_dpp<0x128>(v[r + 4]);
    v[r] = b3 ? x1 : x0;
  }
  // lane bit 2: row_ror:N delivers lane (i - N) mod 16, so the partner i + 4
  // of a lane with bit 2 clear comes from rotate 12 and i - 4 from rotate 4
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const float x0 = fmax_dpp<0x12C>(v[r]), x1 = fmax_dpp<0x124>(v[r + 2]);
    v[r] = b2 ? x1 : x0;
  }
  // lane bit 1 (quad permute [2,3,0,1])
  {
    const float x0 = fmax_dpp<0x4E>(v[0]), x1 = fmax_dpp<0x4E>(v[1]);
    v[0] = b1 ? x1 : x0;
  }
  // lane bit 0 (quad permute [1,0,3,2])
  v[0] = fmax_dpp<0xB1>(v[0]);
  if ((lane & 1) == 0) R[w * ROW_BLOCK + (lane >> 1)] = v[0];
}

// ---------------------------------------------------------- kernels ---

// Rate statistics of row t after the interval (threads t < DK): s^, r, the
// weight Gamma^ (or the given window weight) and the stored rate codes.
template <int DK>
__device__ __forceinline__ void row_rates(const KParams& p, int bh, StatSmem<DK>& st, double m_run,
                                          double e_run, int t) {
  if (t < DK) {
    const double s_hat = -0.5 * log(m_run);
    const double r = 0.5 * e_run;
    st.gam[t] = p.gamma ? p.gamma[(size_t)bh * DK + t] : mode_gamma(p.weight_mode, s_hat, r, p.wb_C);
    p.ws_zr[(size_t)bh * DK + t] = (uint32_t)logq_encode(s_hat) | ((uint32_t)r_encode(r) << 16);
  }
}

// Decode steps of heads with d_k <= 128 hand the requantisation the token's
// vectors (a, g, w) instead of the float32 state; it rebuilds the state from
// the record (d_k = 256 would need a larger LDS staging than its code tile).
constexpr bool compact_decode(int dk) { return dk <= 128; }

// LDS of the statistics pass of one head; the record's code words follow it
// in the same allocation (and, for the per-head budget, the allocator's
// scratch once the words are decoded).
template <int DK, int DV>
struct StatsLds {
  MetaSmem<DK> meta;
  RowSmem<DK> rs;
  __align__(16) StatSmem<DK> st;
};

// Bytes of the code-word staging area that follows StatsLds.  The
// recurrence's partials reuse it once the words are decoded (so a block needs
// less LDS and more blocks fit a compute unit), and so does the per-head
// allocator after the recurrence.
__host__ __device__ inline size_t stats_words_bytes(int wc, int dv) {
  return (size_t)(wc + 1) * dv * 4;
}
template <int DK, int DV>
inline size_t stats_dyn_bytes(int wc) {
  const size_t w = stats_words_bytes(wc, DV);
  return w > sizeof(RecSmem<DK, DV>) ? w : sizeof(RecSmem<DK, DV>);
}

// Decode token tok0 of one head with the state resident in registers,
// starting from the record: the output o, the token's vectors (d_k <= 128) or
// the float32 state after it (d_k = 256) for the requantisation, row ranges
// and EMA rates, weights c and, for the per-head scope, the widths (with
// alloc_sm as the allocator's LDS).  All threads of the block (2 d_k) call it.
template <int DK, int DV, bool HEAD, bool BF16, bool COMPACT>
__device__ __forceinline__ void stats_head(const KParams& p, int bh, StatsLds<DK, DV>& sm,
                                           uint32_t* words, AllocSmem* alloc_sm) {
  const int t = threadIdx.x;
  const int b = bh / p.H, h = bh % p.H;
  const Layout L = p.L;
  const uint8_t* rec = slot_ptr(p.records, L.slot, bh);
  MetaSmem<DK>& meta = sm.meta;
  StatSmem<DK>& st = sm.st;
  // the first token's row scalars are requested with the metadata; the
  // record's meaningful code words (ceil(sum b / 32) per column) follow once
  // the widths are known
  RowIn in = load_rows<DK, BF16>(sm.rs, p, bh, p.tok0);
  load_meta<DK, DV>(rec, L, p.bmax, meta);
  // up to four 16-byte loads per thread are issued now and written to LDS
  // after the row threads' float64 work below, the rest (means above 8 bits
  // at d = 128) then
  constexpr int NPT = 4;
  const int n4 = ((meta.P[DK] + 31) >> 5) * (DV / 4);
  const uint4* wsrc = (const uint4*)(rec + L.codes_off);
  uint4 wv[NPT];
#pragma unroll
  for (int u = 0; u < NPT; ++u) {
    const int e = t + u * (int)blockDim.x;
    wv[u] = e < n4 ? wsrc[e] : make_uint4(0u, 0u, 0u, 0u);
  }
  // EMA states of row t (threads t < DK): from the record, or fresh; token
  // samples are folded in as soon as the token's inputs are loaded (float64
  // work of the row threads that overlaps the other waves' decoding)
  bool fresh = meta.ntok == 0;
  double m_run = 0.0, e_run = 0.0;
  if (t < DK && !fresh) {
    m_run = exp(-2.0 * logq_decode(meta.z[t]));
    e_run = 2.0 * (double)f16_to_f32(meta.r16[t]);
  }
  auto ema = [&](const RowIn& x) {
    if (t < DK) {
      const double zs = decay_sample(x.s), ys = p.no_erase ? 0.0 : erase_sample(x.k, x.beta);
      if (fresh) {
        m_run = zs;
        e_run = ys;
      } else {
        m_run = p.one_minus_alpha * m_run + p.alpha * zs;
        e_run = p.one_minus_alpha * e_run + p.alpha * ys;
      }
    }
    fresh = false;
  };
  ema(in);
  // the step's rates and weights (float64 chains of the row threads) while
  // the code words are in flight
  row_rates<DK>(p, bh, st, m_run, e_run, t);
#pragma unroll
  for (int u = 0; u < NPT; ++u) {
    const int e = t + u * (int)blockDim.x;
    if (e < n4) ((uint4*)words)[e] = wv[u];
  }
  for (int e = t + NPT * (int)blockDim.x; e < n4; e += blockDim.x) ((uint4*)words)[e] = wsrc[e];
  __syncthreads();
  float X[ROW_BLOCK][DV / WAVE];
  unpack_cols<DK, DV>(words, meta, X);
  // COMPACT (one token): the requantisation rebuilds the state from the
  // record and the token's vectors a, g, w; else it reads the float32 state
  constexpr bool compact = COMPACT;
  float* hv = p.ws_hv + (size_t)bh * (DV + 2 * DK);
  {
    const int tok = p.tok0;
    __syncthreads();
    if (compact && t < DK) {
      hv[DV + t] = sm.rs.ak[t].x;        // a = fl32(exp(-s))
      hv[DV + DK + t] = sm.rs.gq[t].x;   // g = fl32(beta k)
    }
    const size_t th = ((size_t)b * p.T + tok) * p.H + h;
    // the words are decoded (barrier above): their space holds the partials
    recur_token<DK, DV, BF16>(X, sm.rs, *(RecSmem<DK, DV>*)words, p.v, th * DV, p.o + th * DV, !p.no_erase,
                              compact ? hv : nullptr);
  }
  if (!compact) {
    // float32 state after the last token, row-major, for the requantisation
    const int w = t / WAVE, lane = lane_id();
    float* dstS = p.ws_s32 + (size_t)bh * DK * DV;
#pragma unroll
    for (int r = 0; r < ROW_BLOCK; ++r)
#pragma unroll
      for (int c = 0; c < DV / WAVE; ++c) dstS[(w * ROW_BLOCK + r) * DV + lane + WAVE * c] = X[r][c];
  }
  row_max<DK, DV>(X, st.R);
  __syncthreads();
  if (p.G > DK) {
    // groups spanning heads: the allocation pass forms R~ over the group
    if (t < DK) {
      p.ws_rpart[(size_t)bh * DK + t] = st.R[t];
      p.ws_gam[(size_t)bh * DK + t] = st.gam[t];
    }
    return;
  }
  row_weights<DK>(p, bh, st, t);
  if constexpr (HEAD) {
    // per-head budget: allocate here (c of this head is in LDS)
    block_allocate<1>([&](int n) { return st.c[n]; }, DK, p.need, p.bmin, p.bmax,
                      p.ws_bits + (size_t)bh * DK, *alloc_sm);
  }
}

template <int DK, int DV, bool HEAD, bool BF16>
__global__ void __launch_bounds__(2 * DK) __attribute__((amdgpu_waves_per_eu(6))) k_chunk(KParams p) {
  extern __shared__ uint4 dyn_lds[];
  __shared__ StatsLds<DK, DV> sm;
  uint32_t* words = (uint32_t*)dyn_lds;
  stats_head<DK, DV, HEAD, BF16, compact_decode(DK)>(p, blockIdx.x, sm, words, (AllocSmem*)dyn_lds);
}

// Layer budget: one block per scope unit of N rows (contiguous in ws_c).
__global__ void __launch_bounds__(1024) k_alloc(const double* c, int N, int need, int bmin,
                                                int bmax, uint8_t* bits) {
  __shared__ AllocSmem sm;
  const double* cu = c + (size_t)blockIdx.x * N;
  block_allocate<ALLOC_MAX_N / 1024>([&](int n) { return cu[n]; }, N, need, bmin, bmax,
                                     bits + (size_t)blockIdx.x * N, sm);
}

template <int DK, int DV, bool COMPACT, bool C8, int PAIRS = 1, int PARTS = 1, bool ALLOC = false>
__global__ void __launch_bounds__(requant_threads(DK, DV, PAIRS, PARTS))
    __attribute__((amdgpu_waves_per_eu(4))) k_requant(KParams p) {
  __shared__ RequantLds<DK, DV, COMPACT, CodeTile<C8>> sm;
  // the parts of a head run on the XCD of the kernels before and after it
  // (one block per head or per column slice of a head, dealt the same way),
  // so the float32 state it reads and the record it writes stay in one L2
  int bh = blockIdx.x, part = 0;
  if constexpr (PARTS > 1) slice_block(p.B * p.H, PARTS, bh, part);
  requant_head<DK, DV, COMPACT, CodeTile<C8>, PAIRS, PARTS, ALLOC>(p, bh, sm, part);
}

// Buffer resource over n bytes at base (word 3 of a gfx9 resource: untyped
// 32-bit data); loads past n return 0 and stores past n are dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(void* base, int n) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, n, 0x00020000);
}
constexpr int BUF_NT = 2;   // cache policy of a buffer access: nontemporal

// Unquantised ("32-bit") state: load, the interval's tokens, store.  Columns
// are independent in the recurrence, so a block takes one 64-column slice of a
// head (blockIdx.x = head * slices + slice): 32 state values per lane keep the
// register count low (eight waves per SIMD for one token, ONE: the decode
// step), and the grid holds more, smaller blocks, which keeps more of the
// state streaming.
template <int DK, int DV, bool BF16, bool ONE>
__global__ void __launch_bounds__(2 * DK) k_step32(KParams p) {
  constexpr int NSL = DV / SLICE;
  const int bh = blockIdx.x / NSL, col0 = (blockIdx.x % NSL) * SLICE;
  const int b = bh / p.H, h = bh % p.H;
  const int w = threadIdx.x / WAVE, lane = lane_id();
  // buffer addressing: the head's state as one resource, the lane's column as
  // the only vector offset, the wave's row as a scalar one (plain 64-bit
  // addresses cost two registers per row in flight)
  const __amdgpu_buffer_rsrc_t S =
      buf_rsrc((uint8_t*)p.records + (long long)bh * DK * DV * 4, DK * DV * 4);
  const int voff = (col0 + lane) * 4;
  const int soff = __builtin_amdgcn_readfirstlane(w) * ROW_BLOCK * DV * 4;
  __shared__ RowSmem<DK> rs;
  __shared__ RecSmem<DK, SLICE> rsm;
  float X[ROW_BLOCK][1];
  for (int j = 0; j < (ONE ? 1 : p.ntk); ++j) {
    const int tok = p.tok0 + j;
    load_rows<DK, BF16>(rs, p, bh, tok);
    // first token: the state is loaded after the row scalars, so that the
    // registers of their float64 exponentials are free again
    if (j == 0) {
#pragma unroll
      for (int r = 0; r < ROW_BLOCK; ++r)
        X[r][0] = __uint_as_float(
            __builtin_amdgcn_raw_buffer_load_b32(S, voff, soff + r * DV * 4, BUF_NT));
    }
    __syncthreads();
    const size_t th = ((size_t)b * p.T + tok) * p.H + h;
    recur_token<DK, SLICE, BF16>(X, rs, rsm, p.v, th * DV + col0, p.o + th * DV + col0,
                                 !p.no_erase);
  }
#pragma unroll
  for (int r = 0; r < ROW_BLOCK; ++r)
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(X[r][0]), S, voff, soff + r * DV * 4,
                                          BUF_NT);
}

// Standalone codec: quantise given states.
template <int DK, int DV>
__global__ void __launch_bounds__(2 * DK) k_pack(KParams p, const float* S, const uint8_t* bits,
                                                 const double* s_hat, const double* r,
                                                 unsigned ntok) {
  const int bh = blockIdx.x;
  const Layout L = p.L;
  uint8_t* rec = (uint8_t*)p.records + L.slot * (long long)bh;
  __shared__ __align__(16) CodeT<DK> Ct[DV * CT_LD_OF<DK>];
  __shared__ __align__(16) uint8_t nb[DK];
  __shared__ uint8_t perm[DK];
  __shared__ uint16_t sc16[DK], zz[DK], rr[DK];
  __shared__ float phi[MAX_B + 1][N_FIT];
  __shared__ OrderSmem<DK> os;
  __shared__ uint32_t tail[DV];
  const int t = threadIdx.x;
  if (t < DK) {
    nb[t] = (uint8_t)min(max((int)bits[(size_t)bh * DK + t], 1), p.bmax);
    zz[t] = logq_encode(s_hat[(size_t)bh * DK + t]);
    rr[t] = r_encode(r[(size_t)bh * DK + t]);
  }
  for (int e = t; e < (MAX_B + 1) * N_FIT; e += blockDim.x) phi[e / N_FIT][e % N_FIT] = p.phi[e / N_FIT][e % N_FIT];
  __syncthreads();
  width_order<DK>(nb, perm, os);
  const float* Sh = S + (size_t)bh * DK * DV;
  fit_rows<DK, DV>([&](int i, int sg, float (&x)[SEG]) { load_dense<DV>(Sh, i, sg, x); }, nb, perm,
                   phi, Ct, sc16, p.diag_fit);
  __syncthreads();
  pack_cols<DK, DV>(Ct, nb, os.P, (uint32_t*)(rec + L.codes_off), tail);
  store_meta<DK>(rec, L, ntok, nb, sc16, zz, rr);
}

// Standalone codec: decode records.
template <int DK, int DV>
__global__ void __launch_bounds__(2 * DK) k_unpack(KParams p, float* S, uint8_t* bits,
                                                   double* s_hat, double* r) {
  constexpr int CPL = DV / WAVE;
  const int bh = blockIdx.x;
  const int t = threadIdx.x, w = t / WAVE, lane = lane_id();
  const Layout L = p.L;
  if (p.state32) {
    if (S) {
      const float* src = (const float*)((const uint8_t*)p.records + (long long)bh * DK * DV * 4);
      for (int e = t; e < DK * DV; e += blockDim.x) S[(size_t)bh * DK * DV + e] = src[e];
    }
    return;
  }
  const uint8_t* rec = slot_ptr(p.records, L.slot, bh);
  __shared__ MetaSmem<DK> meta;
  load_meta<DK, DV>(rec, L, p.bmax, meta);
  extern __shared__ uint4 dyn_lds[];
  stage_words<DV>(rec, L, meta.P[DK], (uint32_t*)dyn_lds);
  if (S) {
    float X[ROW_BLOCK][CPL];
    unpack_cols<DK, DV>((const uint32_t*)dyn_lds, meta, X);
#pragma unroll
    for (int rr_ = 0; rr_ < ROW_BLOCK; ++rr_)
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        S[((size_t)bh * DK + w * ROW_BLOCK + rr_) * DV + lane + WAVE * c] = X[rr_][c];
  }
  if (t < DK) {
    if (bits) bits[(size_t)bh * DK + t] = meta.w[t];
    if (s_hat) s_hat[(size_t)bh * DK + t] = logq_decode(meta.z[t]);
    if (r) r[(size_t)bh * DK + t] = (double)f16_to_f32(meta.r16[t]);
  }
}

// ------------------------------------------ prefill: column slices ---
//
// A prefill chunk (tokens [tok0, tok0 + ntk)) runs d_v / 64 blocks per head,
// one per 64-column slice: the recurrence couples the rows of a column but
// never two columns, so the slices are independent until the write-back.
// Each block keeps its d_k x 64 slice in registers (wave w: rows 32w..32w+31,
// lane: column) and stages the row scalars of PF_TS tokens at a time in LDS,
// the float64 exponentials of all (token, row) pairs computed by all threads.
// It synchronises once per token (partial sums of u double-buffered by token
// parity) and combines the outputs of the staged tokens together.  Slice 0
// also carries the EMA statistics.  Row maxima leave per slice;
// k_alloc_slices combines them into the weights and allocates.

template <int DK>
constexpr int pf_tokens() { return DK > 128 ? 8 : 16; }

template <int DK>
struct PfSmem {
  static constexpr int TS = pf_tokens<DK>();
  static constexpr int NW = DK / ROW_BLOCK;
  float4 rq[TS][DK];        // {fl32(exp(-s)), k, fl32(beta k), q} of (token, row)
  double z[TS][DK];         // exp(-2 s): EMA decay samples (slice 0)
  float beta[TS];
  float v[TS][SLICE];
  float up[2][NW][SLICE];   // partial sums of u, by token parity
  float op[TS][NW][SLICE];  // partial sums of o
};

// One token on a slice (lane = column): the column-layout recurrence with
// the row scalars of staged token j.  One barrier (before the u combine).
template <int DK>
__device__ __forceinline__ void recur_slice(float (&X)[ROW_BLOCK][1], PfSmem<DK>& ps, int j,
                                            bool erase) {
  const int w = threadIdx.x / WAVE, lane = lane_id();
  const float4 s0 = ps.rq[j][w * ROW_BLOCK + (lane & 15)];
  const float4 s1 = ps.rq[j][w * ROW_BLOCK + 16 + (lane & 15)];
  float acc = 0.f;
  pass1_16<0, 0, 1>(X, acc, s0.x, s0.y);
  pass1_16<16, 0, 1>(X, acc, s1.x, s1.y);
  ps.up[j & 1][w][lane] = acc;
  __syncthreads();
  const float u = combine_col<DK, SLICE>(ps.up[j & 1], lane);
  const float wv = erase ? ps.v[j][lane] - u : ps.v[j][lane];   // no erasure: w = v
  acc = 0.f;
  pass2_16<0, 0, 1>(X, acc, s0.z, s0.w, wv);
  pass2_16<16, 0, 1>(X, acc, s1.z, s1.w, wv);
  ps.op[j][w][lane] = acc;
}

template <int DK, bool BF16>
__global__ void __launch_bounds__(2 * DK) k_chunk_slices(KParams p) {
  constexpr int TS = pf_tokens<DK>();
  const int nsl = p.dv / SLICE;
  int bh, sl;
  slice_block(p.B * p.H, nsl, bh, sl);   // a head's slices on one XCD
  const int t = threadIdx.x;
  const int b = bh / p.H, h = bh % p.H;
  const Layout L = p.L;
  const uint8_t* rec = slot_ptr(p.records, L.slot, bh);
  __shared__ MetaSmem<DK> meta;
  __shared__ PfSmem<DK> ps;
  __shared__ float Rrow[DK];
  extern __shared__ uint4 dyn_lds[];
  uint32_t* words = (uint32_t*)dyn_lds;
  {
    // the slice's code words: word kw of column sl*64 + c at words[kw*64 + c]
    const uint4* src = (const uint4*)(rec + L.codes_off);
    constexpr int Q = SLICE / 4;
    const int n4 = L.wc * Q;
    for (int e = t; e < n4; e += blockDim.x)
      ((uint4*)words)[e] = src[(size_t)(e / Q) * (p.dv / 4) + sl * Q + e % Q];
  }
  load_meta<DK, SLICE>(rec, L, p.bmax, meta);   // its barrier covers the staging
  float X[ROW_BLOCK][1];
  unpack_cols<DK, SLICE>(words, meta, X);
  const bool ema_here = sl == 0 && t < DK;
  const bool fresh0 = meta.ntok == 0;
  double m_run = 0.0, e_run = 0.0;
  if (ema_here && !fresh0) {
    m_run = exp(-2.0 * logq_decode(meta.z[t]));
    e_run = 2.0 * (double)f16_to_f32(meta.r16[t]);
  }
  for (int j0 = 0; j0 < p.ntk; j0 += TS) {
    const int nt = min(TS, p.ntk - j0);
    __syncthreads();   // the previous tokens' readers are done with the tables
    {
      // thread t stages row t % DK of tokens 2q + t / DK (all loads first)
      constexpr int NQ = TS / 2;
      const int i = t % DK, jt = t / DK;
      float sv[NQ], kv[NQ], qv[NQ], bt[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int j = 2 * q + jt;
        const size_t th = ((size_t)b * p.T + p.tok0 + j0 + min(j, nt - 1)) * p.H + h;
        sv[q] = p.per_head ? p.s[th] : p.s[th * DK + i];
        kv[q] = in_f32<BF16>(p.k, th * DK + i);
        qv[q] = in_f32<BF16>(p.q, th * DK + i);
        bt[q] = p.beta[th];
      }
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int j = 2 * q + jt;
        if (j < nt) {
          ps.rq[j][i] = make_float4((float)exp(-(double)sv[q]), kv[q], bt[q] * kv[q], qv[q]);
          if (sl == 0) ps.z[j][i] = decay_sample(sv[q]);
          if (i == 0) ps.beta[j] = bt[q];
        }
      }
    }
    for (int e = t; e < nt * SLICE; e += blockDim.x) {
      const int j = e / SLICE, c = e % SLICE;
      const size_t th = ((size_t)b * p.T + p.tok0 + j0 + j) * p.H + h;
      ps.v[j][c] = in_f32<BF16>(p.v, th * p.dv + sl * SLICE + c);
    }
    __syncthreads();
    if (ema_here) {
      // token-sequential EMA of row t (the first token initialises a fresh record)
      for (int j = 0; j < nt; ++j) {
        const double zs = ps.z[j][t];
        const double ys = p.no_erase ? 0.0 : erase_sample(ps.rq[j][t].y, ps.beta[j]);
        if (fresh0 && j0 + j == 0) {
          m_run = zs;
          e_run = ys;
        } else {
          m_run = p.one_minus_alpha * m_run + p.alpha * zs;
          e_run = p.one_minus_alpha * e_run + p.alpha * ys;
        }
      }
    }
    for (int j = 0; j < nt; ++j) recur_slice<DK>(X, ps, j, !p.no_erase);
    __syncthreads();
    for (int e = t; e < nt * SLICE; e += blockDim.x) {
      const int j = e / SLICE, c = e % SLICE;
      const size_t th = ((size_t)b * p.T + p.tok0 + j0 + j) * p.H + h;
      p.o[th * p.dv + sl * SLICE + c] = combine_col<DK, SLICE>(ps.op[j], c);
    }
  }
  {
    // float32 state after the chunk (this slice's columns), row-major
    const int w = t / WAVE, lane = lane_id();
    float* dstS = p.ws_s32 + (size_t)bh * DK * p.dv + sl * SLICE;
#pragma unroll
    for (int r = 0; r < ROW_BLOCK; ++r) dstS[(size_t)(w * ROW_BLOCK + r) * p.dv + lane] = X[r][0];
  }
  row_max<DK, SLICE>(X, Rrow);
  __syncthreads();
  if (t < DK) p.ws_rpart[((size_t)bh * DK + t) * nsl + sl] = Rrow[t];
  if (ema_here) {
    const double s_hat = -0.5 * log(m_run);
    const double r = 0.5 * e_run;
    p.ws_gam[(size_t)bh * DK + t] = p.gamma ? p.gamma[(size_t)bh * DK + t] : mode_gamma(p.weight_mode, s_hat, r, p.wb_C);
    p.ws_zr[(size_t)bh * DK + t] = (uint32_t)logq_encode(s_hat) | ((uint32_t)r_encode(r) << 16);
  }
}

// ------------------------------------- prefill: row blocks in one wave ---
//
// The same chunk on 64-column slices for d_k <= 128, with the d_k / 32 row
// blocks of a column held by one wave: lane l of wave w has row block
// rb = l / CPW and slice column w * CPW + l % CPW (CPW = 64 / (d_k / 32)
// columns per wave), rows 32 rb .. 32 rb + 31 in registers.  The partial sums
// of a column's row blocks meet inside the wave: permlane32 swaps pair row
// blocks rb and rb + 2 (or rb + 1 when there are two), permlane16 swaps then
// pair rb and rb + 1, the contract's halving order with the same operands.
// So a token needs no barrier; row scalars still reach the lanes by DPP
// row broadcasts (a 16-lane DPP row lies inside one row block).

// Sum of the partials of the row blocks of a column (see above); every lane
// of the column receives the total.
template <int NRB>
__device__ __forceinline__ float rowblock_sum(float x) {
  static_assert(NRB == 2 || NRB == 4, "row blocks per wave");
  const int xi = __builtin_bit_cast(int, x);
  const auto a = __builtin_amdgcn_permlane32_swap(xi, xi, false, false);
  x = __builtin_bit_cast(float, (int)a[0]) + __builtin_bit_cast(float, (int)a[1]);
  if constexpr (NRB == 4) {
    const int yi = __builtin_bit_cast(int, x);
    const auto c = __builtin_amdgcn_permlane16_swap(yi, yi, false, false);
    x = __builtin_bit_cast(float, (int)c[0]) + __builtin_bit_cast(float, (int)c[1]);
  }
  return x;
}

// Maximum over the CPW lanes of a row block (every lane receives it).
template <int CPW>
__device__ __forceinline__ float rowblock_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));    // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_f<0x4E>(v));    // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_f<0x141>(v));   // row_half_mirror
  v = fmaxf(v, dpp_f<0x140>(v));   // row_mirror: the 16-lane row's maximum
  if constexpr (CPW == 32) {
    const int vi = __builtin_bit_cast(int, v);
    const auto c = __builtin_amdgcn_permlane16_swap(vi, vi, false, false);
    v = fmaxf(__builtin_bit_cast(float, (int)c[0]), __builtin_bit_cast(float, (int)c[1]));
  }
  return v;
}

template <int DK>
struct PcSmem {
  static constexpr int TS = 16;
  static constexpr int NRB = DK / ROW_BLOCK;
  float4 rq[TS][DK];        // {fl32(exp(-s)), k, fl32(beta k), q} of (token, row)
  double z[TS][DK];         // exp(-2 s): EMA decay samples (slice 0)
  float beta[TS];
  float v[TS][SLICE];
  float o[TS][SLICE];
  float Rw[NRB][DK];        // row maxima of each wave's columns
};

template <int DK, bool BF16>
__global__ void __launch_bounds__(2 * DK) k_chunk_cols(KParams p) {
  constexpr int NRB = DK / ROW_BLOCK;       // row blocks = waves per block
  constexpr int CPW = WAVE / NRB;           // columns per wave
  constexpr int TS = PcSmem<DK>::TS;
  constexpr int NQ = TS / 2;                // tokens staged per thread and batch
  constexpr int NV = TS * SLICE / (2 * DK); // values of v staged per thread and batch
  static_assert(NRB * CPW == SLICE && CPW >= 16, "16-lane DPP rows inside a row block");
  const int nsl = p.dv / SLICE;
  int bh, sl;
  slice_block(p.B * p.H, nsl, bh, sl);   // a head's slices on one XCD
  const int t = threadIdx.x, w = t / WAVE, lane = lane_id();
  const int rb = lane / CPW, col = w * CPW + lane % CPW;   // slice-local column
  const int b = bh / p.H, h = bh % p.H;
  const Layout L = p.L;
  const uint8_t* rec = slot_ptr(p.records, L.slot, bh);
  __shared__ MetaSmem<DK> meta;
  __shared__ PcSmem<DK> ps;
  extern __shared__ uint4 dyn_lds[];
  uint32_t* words = (uint32_t*)dyn_lds;
  // token inputs of one batch in registers: thread t holds row t % DK of
  // tokens 2q + t / DK, and NV values of v; the next batch's loads are in
  // flight while the current batch runs
  const int si = t % DK, sj = t / DK;
  float sv[NQ], kv[NQ], qv[NQ], bt[NQ], vv[NV];
  auto issue = [&](int j0) {
    const int nt = min(TS, p.ntk - j0);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int j = 2 * q + sj;
      const size_t th = ((size_t)b * p.T + p.tok0 + j0 + min(j, nt - 1)) * p.H + h;
      sv[q] = p.per_head ? p.s[th] : p.s[th * DK + si];
      kv[q] = in_f32<BF16>(p.k, th * DK + si);
      qv[q] = in_f32<BF16>(p.q, th * DK + si);
      bt[q] = p.beta[th];
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int e = t + u * (2 * DK), j = e / SLICE, c = e % SLICE;
      const size_t th = ((size_t)b * p.T + p.tok0 + j0 + min(j, nt - 1)) * p.H + h;
      vv[u] = in_f32<BF16>(p.v, th * p.dv + sl * SLICE + c);
    }
  };
  auto stage = [&](int nt) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int j = 2 * q + sj;
      if (j < nt) {
        ps.rq[j][si] = make_float4((float)exp(-(double)sv[q]), kv[q], bt[q] * kv[q], qv[q]);
        if (sl == 0) ps.z[j][si] = decay_sample(sv[q]);
        if (si == 0) ps.beta[j] = bt[q];
      }
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int e = t + u * (2 * DK);
      ps.v[e / SLICE][e % SLICE] = vv[u];
    }
  };
  auto write_o = [&](int j0, int nt) {
    for (int e = t; e < nt * SLICE; e += blockDim.x) {
      const int j = e / SLICE, c = e % SLICE;
      const size_t th = ((size_t)b * p.T + p.tok0 + j0 + j) * p.H + h;
      p.o[th * p.dv + sl * SLICE + c] = ps.o[j][c];
    }
  };
  if (p.ntk > 0) issue(0);
  {
    // the slice's code words: word kw of column sl*64 + c at words[kw*64 + c]
    const uint4* src = (const uint4*)(rec + L.codes_off);
    constexpr int Q = SLICE / 4;
    const int n4 = L.wc * Q;
    for (int e = t; e < n4; e += blockDim.x)
      ((uint4*)words)[e] = src[(size_t)(e / Q) * (p.dv / 4) + sl * Q + e % Q];
  }
  load_meta<DK, SLICE>(rec, L, p.bmax, meta);   // its barrier covers the staging
  float X[ROW_BLOCK][1];
  // decode rows 32 rb + r of this lane's column: descriptors per lane (the
  // row blocks of a wave differ), x^ = (code + add) mul as in unpack_cols
#pragma unroll
  for (int r = 0; r < ROW_BLOCK; ++r) {
    const uint4 d = meta.desc[rb * ROW_BLOCK + r];
    const int sh = (int)(d.y & 31u), bw = (int)(d.y >> 8);
    const uint32_t lo = words[d.x + col], hi = words[d.x + SLICE + col];
    const int code = __builtin_amdgcn_sbfe((int)__builtin_amdgcn_alignbit(hi, lo, (uint32_t)sh), 0, bw);
    X[r][0] = ((float)code + __builtin_bit_cast(float, d.w)) * __builtin_bit_cast(float, d.z);
  }
  const bool ema_here = sl == 0 && t < DK;
  const bool fresh0 = meta.ntok == 0;
  double m_run = 0.0, e_run = 0.0;
  if (ema_here && !fresh0) {
    m_run = exp(-2.0 * logq_decode(meta.z[t]));
    e_run = 2.0 * (double)f16_to_f32(meta.r16[t]);
  }
  const bool erase = !p.no_erase;
  int prev0 = 0, prevn = 0;
  for (int j0 = 0; j0 < p.ntk; j0 += TS) {
    const int nt = min(TS, p.ntk - j0);
    __syncthreads();   // the previous batch's readers are done with the tables
    if (prevn > 0) write_o(prev0, prevn);
    stage(nt);
    if (j0 + TS < p.ntk) issue(j0 + TS);
    __syncthreads();
    if (ema_here) {
      // token-sequential EMA of row t (the first token initialises a fresh record)
      for (int j = 0; j < nt; ++j) {
        const double zs = ps.z[j][t];
        const double ys = erase ? erase_sample(ps.rq[j][t].y, ps.beta[j]) : 0.0;
        if (fresh0 && j0 + j == 0) {
          m_run = zs;
          e_run = ys;
        } else {
          m_run = p.one_minus_alpha * m_run + p.alpha * zs;
          e_run = p.one_minus_alpha * e_run + p.alpha * ys;
        }
      }
    }
    // rows 32 rb + lane % 16 and 32 rb + 16 + lane % 16: DPP broadcast sources.
    // The batch's first token runs its first pass alone; every later token's
    // first pass is fused with the previous token's second pass (fused_pass),
    // and the batch's last token runs its second pass alone.
    float4 s0 = ps.rq[0][rb * ROW_BLOCK + (lane & 15)];
    float4 s1 = ps.rq[0][rb * ROW_BLOCK + 16 + (lane & 15)];
    float accU = 0.f;
    pass1_16<0, 0, 1>(X, accU, s0.x, s0.y);
    pass1_16<16, 0, 1>(X, accU, s1.x, s1.y);
    for (int j = 0; j + 1 < nt; ++j) {
      const float vj = ps.v[j][col];
      const float4 n0 = ps.rq[j + 1][rb * ROW_BLOCK + (lane & 15)];
      const float4 n1 = ps.rq[j + 1][rb * ROW_BLOCK + 16 + (lane & 15)];
      const float u = rowblock_sum<NRB>(accU);
      const float wv = erase ? vj - u : vj;   // no erasure: w = v
      float accO = 0.f;
      accU = 0.f;
      fused_pass(X, accO, accU, s0.z, s0.w, n0.x, n0.y, s1.z, s1.w, n1.x, n1.y, wv);
      s0 = n0;
      s1 = n1;
      const float o = rowblock_sum<NRB>(accO);
      if (rb == 0) ps.o[j][col] = o;
    }
    {
      const float vj = ps.v[nt - 1][col];
      const float u = rowblock_sum<NRB>(accU);
      const float wv = erase ? vj - u : vj;
      float accO = 0.f;
      pass2_16<0, 0, 1>(X, accO, s0.z, s0.w, wv);
      pass2_16<16, 0, 1>(X, accO, s1.z, s1.w, wv);
      const float o = rowblock_sum<NRB>(accO);
      if (rb == 0) ps.o[nt - 1][col] = o;
    }
    prev0 = j0;
    prevn = nt;
  }
  __syncthreads();
  write_o(prev0, prevn);
  {
    // float32 state after the chunk (this lane's column), row-major
    float* dstS = p.ws_s32 + (size_t)bh * DK * p.dv + sl * SLICE + col;
#pragma unroll
    for (int r = 0; r < ROW_BLOCK; ++r) dstS[(size_t)(rb * ROW_BLOCK + r) * p.dv] = X[r][0];
  }
  // row maxima over the slice: the wave's columns, then the waves
#pragma unroll
  for (int r = 0; r < ROW_BLOCK; ++r) {
    const float m = rowblock_max<CPW>(fabsf(X[r][0]));
    if (lane % CPW == 0) ps.Rw[w][rb * ROW_BLOCK + r] = m;
  }
  __syncthreads();
  if (t < DK) {
    float m = ps.Rw[0][t];
#pragma unroll
    for (int q = 1; q < NRB; ++q) m = fmaxf(m, ps.Rw[q][t]);
    p.ws_rpart[((size_t)bh * DK + t) * nsl + sl] = m;
  }
  if (ema_here) {
    const double s_hat = -0.5 * log(m_run);
    const double r = 0.5 * e_run;
    p.ws_gam[(size_t)bh * DK + t] = p.gamma ? p.gamma[(size_t)bh * DK + t] : mode_gamma(p.weight_mode, s_hat, r, p.wb_C);
    p.ws_zr[(size_t)bh * DK + t] = (uint32_t)logq_encode(s_hat) | ((uint32_t)r_encode(r) << 16);
  }
}

// Weights of the rows of one scope unit from row maxima (given per slice:
// Rp[row][nsl]) and Gamma (group RMS of G consecutive rows in float64, rows
// summed in order; groups may span heads), then the allocation into bits.
__global__ void __launch_bounds__(1024) k_alloc_slices(KParams p, int N, int nsl, const float* Rp,
                                                       const double* gam, uint8_t* bits) {
  __shared__ AllocSmem sm;
  __shared__ __align__(16) float R[ALLOC_MAX_N];
  __shared__ double rms[ALLOC_MAX_N];
  __shared__ double c[ALLOC_MAX_N];
  const int tid = threadIdx.x, nt = blockDim.x;
  const size_t row0 = (size_t)blockIdx.x * N;
  // rows n = tid + k nt: their Gamma and per-slice maxima are loaded before
  // anything waits on them
  constexpr int RPT = ALLOC_MAX_N / 1024;
  constexpr int MAXSL = 4;   // slices per row (d_v <= 256: at most four)
  double gk[RPT];
  float rk[RPT][MAXSL];
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int n = tid + k * nt;
    gk[k] = n < N ? gam[row0 + n] : 0.0;
#pragma unroll
    for (int q = 0; q < MAXSL; ++q) rk[k][q] = n < N && q < nsl ? Rp[(row0 + n) * nsl + q] : 0.f;
  }
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int n = tid + k * nt;
    if (n < N) {
      float m = rk[k][0];
#pragma unroll
      for (int q = 1; q < MAXSL; ++q)
        if (q < nsl) m = fmaxf(m, rk[k][q]);
      R[n] = m;
    }
  }
  __syncthreads();
  const int G = p.G, runs = (G + RMS_RUN - 1) / RMS_RUN;
  // group RMS: squares summed in runs of RMS_RUN rows (each in row order),
  // the run sums (held in c until the weights are formed) added in order
  for (int u = tid; u < (N / G) * runs; u += nt) {
    const int g = u / runs, r0 = g * G + (u % runs) * RMS_RUN;
    c[u] = run_sumsq(R, r0, min(r0 + RMS_RUN, (g + 1) * G));
  }
  __syncthreads();
  for (int g = tid; g < N / G; g += nt) {
    double acc = 0.0;
    for (int k = 0; k < runs; ++k) acc = acc + c[g * runs + k];
    rms[g] = sqrt(acc / (double)G);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int n = tid + k * nt;
    if (n < N) c[n] = mode_key(p.weight_mode, gk[k], R[n], rms[n / G]);
  }
  __syncthreads();
  block_allocate<ALLOC_MAX_N / 1024>([&](int n) { return c[n]; }, N, p.need, p.bmin, p.bmax,
                                     bits + row0, sm);
}

// ------------------------------------------------------- launchers ---

// One write-back interval: tokens [p.tok0, p.tok0 + p.ntk), then quantise.
// phases: 1 = stats and allocation, 2 = requantisation, 3 = both.
template <int DK, int DV>
static hipError_t launch_interval_t(const KParams& p, hipStream_t st, int phases = 3) {
  const int nbh = p.B * p.H;
  if (p.state32) {
    if (!(phases & 1)) return hipSuccess;
    const int nblk = nbh * (DV / SLICE);
    if (p.ntk == 1)
      return p.in_bf16 ? launch("step32", k_step32<DK, DV, true, true>, nblk, 2 * DK, 0, st, p)
                       : launch("step32", k_step32<DK, DV, false, true>, nblk, 2 * DK, 0, st, p);
    return p.in_bf16 ? launch("step32", k_step32<DK, DV, true, false>, nblk, 2 * DK, 0, st, p)
                     : launch("step32", k_step32<DK, DV, false, false>, nblk, 2 * DK, 0, st, p);
  }
  hipError_t e = hipSuccess;
  if (phases & 1) {
    // code-word staging; with the per-head budget the allocator's scratch
    // reuses it after the words are decoded
    size_t dyn = stats_dyn_bytes<DK, DV>(p.L.wc);
    if (p.scope == 1 && dyn < sizeof(AllocSmem)) dyn = sizeof(AllocSmem);
    if (p.scope == 1)
      e = p.in_bf16 ? launch("stats", k_chunk<DK, DV, true, true>, nbh, 2 * DK, dyn, st, p)
                    : launch("stats", k_chunk<DK, DV, true, false>, nbh, 2 * DK, dyn, st, p);
    else
      e = p.in_bf16 ? launch("stats", k_chunk<DK, DV, false, true>, nbh, 2 * DK, dyn, st, p)
                    : launch("stats", k_chunk<DK, DV, false, false>, nbh, 2 * DK, dyn, st, p);
    if (e != hipSuccess) return e;
    if (p.scope == 0) {
      if (p.G > DK)   // groups spanning heads: weights from the row maxima and Gamma
        e = launch("alloc", k_alloc_slices, p.B, 1024, 0, st, p, p.H * DK, 1,
                   (const float*)p.ws_rpart, (const double*)p.ws_gam, p.ws_bits);
      else
        e = launch("alloc", k_alloc, p.B, 1024, 0, st, p.ws_c, p.H * DK, p.need, p.bmin, p.bmax,
                   p.ws_bits);
      if (e != hipSuccess) return e;
    }
  }
  if (!(phases & 2)) return hipSuccess;
  if (DK > 128 || p.bmax <= 8)
    return launch("requant", k_requant<DK, DV, compact_decode(DK), true>, nbh, 2 * DK, 0, st, p);
  return launch("requant", k_requant<DK, DV, compact_decode(DK), (DK > 128)>, nbh, 2 * DK, 0, st, p);
}

static hipError_t launch_interval(const KParams& p, hipStream_t st, int phases = 3) {
  if (p.dk == 64) return launch_interval_t<64, 64>(p, st, phases);
  if (p.dk == 256) return launch_interval_t<256, 256>(p, st, phases);
  return launch_interval_t<128, 128>(p, st, phases);
}

hipError_t launch_step(const KParams& p, hipStream_t st) { return launch_interval(p, st); }
hipError_t launch_step_outputs(const KParams& p, hipStream_t st) { return launch_interval(p, st, 1); }
hipError_t launch_step_writeback(const KParams& p, hipStream_t st) {
  return launch_interval(p, st, 2);
}

// One prefill write-back interval on column slices: stats per slice, weights
// and allocation per scope unit, then the requantisation.
template <int DK>
static hipError_t launch_interval_slices(const KParams& p, hipStream_t st) {
  const int nsl = p.dv / SLICE;
  const size_t dyn = (size_t)(p.L.wc + 1) * SLICE * 4;
  hipError_t e;
  if constexpr (DK <= 128)
    e = p.in_bf16 ? launch("stats", k_chunk_cols<DK, true>, p.B * p.H * nsl, 2 * DK, dyn, st, p)
                  : launch("stats", k_chunk_cols<DK, false>, p.B * p.H * nsl, 2 * DK, dyn, st, p);
  else
    e = p.in_bf16 ? launch("stats", k_chunk_slices<DK, true>, p.B * p.H * nsl, 2 * DK, dyn, st, p)
                  : launch("stats", k_chunk_slices<DK, false>, p.B * p.H * nsl, 2 * DK, dyn, st, p);
  if (e != hipSuccess) return e;
  return launch_chunk_writeback(p, nsl, st);
}

static hipError_t launch_chunk_alloc(const KParams& p, int nsl, hipStream_t st, bool keys) {
  const int units = p.scope == 0 ? p.B : p.B * p.H;
  const int N = p.scope == 0 ? p.H * p.dk : p.dk;
  if (keys)
    return launch("alloc", k_alloc, units, 1024, 0, st, p.ws_c, N, p.need, p.bmin, p.bmax, p.ws_bits);
  return launch("alloc", k_alloc_slices, units, 1024, 0, st, p, N, nsl,
                (const float*)p.ws_rpart, (const double*)p.ws_gam, p.ws_bits);
}

static hipError_t launch_chunk_requant(const KParams& p, hipStream_t st) {
  const int DK = p.dk;
  // d_v <= 128: the fit evaluates FL candidates of a row segment at once
  // (FL times the lanes per head; a prefill has few heads, so the grid alone
  // would leave SIMDs idle, and the rows with the longest candidate scans
  // would set the time of the block) and two blocks share each head (rows
  // split in halves)
  constexpr int FL = 4, PT = 2;
  const bool c8 = DK > 128 || p.bmax <= 8;
  constexpr int T64 = requant_threads(64, 64, FL, PT), T128 = requant_threads(128, 128, FL, PT);
  const int nblk = p.B * p.H * PT;
  if (DK == 64)
    return c8 ? launch("requant", k_requant<64, 64, false, true, FL, PT>, nblk, T64, 0, st, p)
              : launch("requant", k_requant<64, 64, false, false, FL, PT>, nblk, T64, 0, st, p);
  if (DK == 256) return launch("requant", k_requant<256, 256, false, true>, p.B * p.H, 512, 0, st, p);
  return c8 ? launch("requant", k_requant<128, 128, false, true, FL, PT>, nblk, T128, 0, st, p)
            : launch("requant", k_requant<128, 128, false, false, FL, PT>, nblk, T128, 0, st, p);
}

hipError_t launch_chunk_writeback(const KParams& p, int nsl, hipStream_t st, bool keys) {
  if (keys && p.dk == 128) {
    // the weights are ready: each requantisation block selects its unit's
    // widths itself (one launch per interval fewer)
    constexpr int FL = 4, PT = 2, T128 = requant_threads(128, 128, FL, PT);
    const int nblk = p.B * p.H * PT;
    return p.bmax <= 8
               ? launch("requant", k_requant<128, 128, false, true, FL, PT, true>, nblk, T128, 0, st, p)
               : launch("requant", k_requant<128, 128, false, false, FL, PT, true>, nblk, T128, 0, st, p);
  }
  const hipError_t e = launch_chunk_alloc(p, nsl, st, keys);
  return e != hipSuccess ? e : launch_chunk_requant(p, st);
}

hipError_t launch_prefill(KParams p, int C, hipStream_t st) {
  if (p.state32) {
    p.tok0 = 0;
    p.ntk = p.T;
    return launch_interval(p, st);
  }
  for (int t0 = 0; t0 < p.T; t0 += C) {
    p.tok0 = t0;
    p.ntk = (p.T - t0) < C ? (p.T - t0) : C;
    hipError_t e;
    if (p.dk == 64)
      e = launch_interval_slices<64>(p, st);
    else if (p.dk == 256)
      e = launch_interval_slices<256>(p, st);
    else
      e = launch_interval_slices<128>(p, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_pack(const KParams& p, const float* S, const uint8_t* bits, const double* s_hat,
                       const double* r, unsigned ntok, hipStream_t st) {
  const int nbh = p.B * p.H;
  if (p.dk == 64) return launch("pack", k_pack<64, 64>, nbh, 128, 0, st, p, S, bits, s_hat, r, ntok);
  if (p.dk == 256)
    return launch("pack", k_pack<256, 256>, nbh, 512, 0, st, p, S, bits, s_hat, r, ntok);
  return launch("pack", k_pack<128, 128>, nbh, 256, 0, st, p, S, bits, s_hat, r, ntok);
}

hipError_t launch_unpack(const KParams& p, float* S, uint8_t* bits, double* s_hat, double* r,
                         hipStream_t st) {
  const int nbh = p.B * p.H;
  const size_t dyn = p.state32 ? 0 : (size_t)(p.L.wc + 1) * p.dv * 4;
  if (p.dk == 64) return launch("unpack", k_unpack<64, 64>, nbh, 128, dyn, st, p, S, bits, s_hat, r);
  if (p.dk == 256)
    return launch("unpack", k_unpack<256, 256>, nbh, 512, dyn, st, p, S, bits, s_hat, r);
  return launch("unpack", k_unpack<128, 128>, nbh, 256, dyn, st, p, S, bits, s_hat, r);
}

hipError_t launch_alloc_bits(const KParams& p, const double* gamma, const float* R, uint8_t* bits,
                             hipStream_t st) {
  const int units = p.scope == 0 ? p.B : p.B * p.H;
  const int N = p.scope == 0 ? p.H * p.dk : p.dk;
  return launch("alloc", k_alloc_slices, units, 1024, 0, st, p, N, 1, R, gamma, bits);
}

}  // namespace kda
