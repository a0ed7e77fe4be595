// Chunked prefill on MFMA: the gated delta rule (eq. rule, Sec. 2) over one
// write-back interval in its WY/UT form.
//
// Within a chunk of n <= 64 tokens starting from the dequantised state S0
// (d_k x d_v), with c_j = sum_{tau<=j} s_tau per row (cumulative decay) and
// gamma_j = exp(-c_j), the substitution S_j = diag(gamma_j) Z_j turns the
// recurrence S_j = (I - beta_j k_j k_j^T) D_j S_{j-1} + beta_j k_j v_j^T
// into Z_j = Z_{j-1} + (k_j / gamma_j) u_j^T with
// u_j = beta_j (v_j - Z_{j-1}^T (gamma_j k_j)); collecting the u_j as rows of
// U gives a unit lower-triangular system, and the outputs and the state at
// the chunk's end follow:
//
//   L[j][tau] = sum_i k_ji k_taui exp(c_taui - c_ji)      (tau < j)
//   A[j][tau] = sum_i q_ji k_taui exp(c_taui - c_ji)      (tau <= j)
//   T         = (I + diag(beta) L)^-1                      (unit lower triangular)
//   U         = T diag(beta) (V - Khat S0),  Khat_j = k_j * gamma_j
//   O         = Qhat S0 + A U,               Qhat_j = q_j * gamma_j
//   S_n       = gamma_{n-1} * S0 + Ktil^T U, Ktil_tau = k_tau * exp(c_tau - c_{n-1})
//
// Without erasure L = 0 and U = diag(beta) V.  Everything but the three
// products with S0 depends on the chunk's inputs only, so it is formed for
// many chunks at once (k_chunk_prep, one block per chunk and head, spread
// over the whole GPU) and stored in a per-chunk record; the write-back loop
// then runs k_chunk_apply (W = Wk S0, U = Uv - W, O, S_n; bf16 MFMA with
// float32 accumulation) followed by the allocation and requantisation
// kernels of the token-sequential path.
//
// The pairwise decay factors are split as exp(c_tau - c_r) exp(c_r - c_j)
// around the last token r of the previous 16-token block, which keeps every
// factor of an off-diagonal block at most 1; a diagonal block whose decay
// span within the block stays below 80 uses the same split (factors within
// [e^-80, e^80], finite in bf16 and float32), otherwise it is formed on the
// vector ALUs with one exponential per pair and row.
//
// EMA statistics over the chunk (Sec. 3, running statistics) are affine in
// their value at the chunk start: m_n = (1 - alpha)^n m_0 + Q with Q the
// same recursion started from 0 (a fresh record starts from m_0 = its first
// sample).  k_chunk_prep forms Q over token segments (each in token order,
// combined in order with the powers of 1 - alpha), k_chunk_apply applies it
// to the record's stored value.  The results differ from the token-order
// recursion by rounding in the last bits of a double.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kda_alloc.hpp"
#include "kda_device.hpp"
#include "kda_kernels.hpp"
#include "kda_profile.hpp"
#include "kda_record.hpp"

namespace kda {

namespace {

constexpr int CT = 64;          // tokens of a (padded) chunk
constexpr int NT = 256;         // threads per apply block: four waves
constexpr int NTP = 512;        // threads per prep block: eight waves
constexpr float SPLIT_SPAN = 80.f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // 16-byte copies held in registers

// float -> bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint16_t bf16_rne(float x) {
  uint32_t u = __builtin_bit_cast(uint32_t, x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_f32(uint16_t h) {
  return __builtin_bit_cast(float, (uint32_t)h << 16);
}

// x = hi + lo with hi = bf16(x) and lo = bf16(x - hi) (x - hi is exact in
// float32): the pair holds x to a relative 2^-18.
__device__ __forceinline__ uint16_t bf16_lo(float x, uint16_t hi) { return bf16_rne(x - bf16_f32(hi)); }

// Two values as packed hi and lo pairs.
__device__ __forceinline__ void split2(float a, float b, uint32_t& hi, uint32_t& lo) {
  const uint16_t ah = bf16_rne(a), bh = bf16_rne(b);
  hi = (uint32_t)ah | ((uint32_t)bh << 16);
  lo = (uint32_t)bf16_lo(a, ah) | ((uint32_t)bf16_lo(b, bh) << 16);
}

// D += A B for 16x16 tiles, K = 32: lane l supplies row l % 16 of A and
// column l % 16 of B, each at k = 8 (l / 16) .. 8 (l / 16) + 7 (eight bf16
// in one 16-byte register quad); it receives D rows 4 (l / 16) + r, r < 4,
// of column l % 16.
__device__ __forceinline__ f32x4 mma(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// D += (Ah + Al)(Bh + Bl) to a relative 2^-17: the three products of the
// split pairs (Al Bl, below 2^-18 of the product, is dropped).
__device__ __forceinline__ f32x4 mma3(uint4 ah, uint4 al, uint4 bh, uint4 bl, f32x4 c) {
  c = mma(al, bh, c);
  c = mma(ah, bl, c);
  return mma(ah, bh, c);
}

// D += (Ah + Al) B for an operand B exact in bf16.
__device__ __forceinline__ f32x4 mma2(uint4 ah, uint4 al, uint4 b, f32x4 c) {
  c = mma(al, b, c);
  return mma(ah, b, c);
}

__device__ __forceinline__ float max16(float m) {
  // maximum over the 16 lanes of a row group (l / 16 fixed)
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 16));
  return m;
}

}  // namespace

// Byte layout of one chunk's record (per chunk and head), 256-byte aligned
// fields; DV == DK.  Matrices that enter MFMA products as the A operand are
// stored as bf16 hi and lo planes (hi = bf16(x), lo = bf16(x - hi)), so the
// products keep float32-level accuracy (three bf16 MFMAs each).
template <int DK>
struct ChunkWs {
  static constexpr size_t PL = (size_t)CT * DK * 2;       // one bf16 [CT][DK] plane
  static constexpr size_t wk = 0;                         // bf16 [2][CT][DK]: T diag(beta) Khat
  static constexpr size_t qh = wk + 2 * PL;               // bf16 [2][CT][DK]: Qhat
  static constexpr size_t ktt = qh + 2 * PL;              // bf16 [2][DK][CT]: Ktil^T
  static constexpr size_t am = ktt + 2 * PL;              // bf16 [2][CT][CT]: A (lower, with diagonal)
  static constexpr size_t uv = am + (size_t)2 * CT * CT * 2;  // f32 [CT][DK]: T diag(beta) V
  static constexpr size_t gend = uv + (size_t)CT * DK * 4;// f32 [DK]: gamma_{n-1}
  static constexpr size_t ema = gend + (size_t)DK * 4;    // f64 [4][DK]: Q_m, Q_e, first samples
  static constexpr size_t gam = ema + (size_t)4 * DK * 8; // f64 [DK]: Gamma after the chunk
  static constexpr size_t zr = gam + (size_t)DK * 8;      // u32 [DK]: rate codes stored after it
  static constexpr size_t bytes = (zr + (size_t)DK * 4 + 255) / 256 * 256;
};

template <int DK>
struct PrepSmem {
  static constexpr int CS = DK + 4;   // float row stride (16-byte aligned rows)
  static constexpr int KS = DK + 8;   // bf16 row stride
  static constexpr int LS = CT + 4;
  static constexpr int TS = CT + 8;
  static constexpr int SEGS = NTP / DK;  // token segments of the decay scan
  union {
    float c[CT][CS];                  // cumulative decay exponents
    struct {
      float T[CT][LS];                // (I + diag(beta) L)^-1
      float X[4][16][20];             // per-wave 16x16 products
      uint16_t tbl[CT][TS];           // lo plane of T diag(beta)
    } t;
  } u0;
  uint16_t k[CT][KS], q[CT][KS];      // keys and queries
  uint16_t vt[DK][TS];                // V^T
  uint16_t kht[2][DK][TS];            // Khat^T, hi and lo planes
  union {
    float L[CT][LS];                  // strictly lower L
    struct {
      float csum[SEGS][DK];           // decay sums of the segments
      double em[SEGS][2][DK];         // EMA sums of the segments (from zero)
      double first[2][DK];            // first samples of the chunk
    } seg;
  } u1;
  uint16_t tb[CT][TS];                // T diag(beta), bf16 hi plane
  float beta[CT];
};

// The state-independent parts of one chunk of one head (unit = chunk of the
// group * B H + head); all threads of the block call it.
template <int DK>
__device__ __forceinline__ void prep_unit(const KParams& p, int C, uint8_t* cws, int unit,
                                          PrepSmem<DK>& sm) {
  using CW = ChunkWs<DK>;
  using SM = PrepSmem<DK>;
  constexpr int SEGS = SM::SEGS, SEGL = CT / SEGS;
  const int nbh = p.B * p.H;
  const int cg = unit / nbh, bh = unit % nbh;
  const int b = bh / p.H, h = bh % p.H;
  const int t = threadIdx.x, w = t / WAVE, lane = lane_id();
  const int tok0 = p.tok0 + cg * C;
  const int n = min(C, p.T - tok0);
  uint8_t* out = cws + ((size_t)cg * nbh + bh) * CW::bytes;
  auto th = [&](int j) { return ((size_t)b * p.T + tok0 + j) * p.H + h; };
  const bool erase = !p.no_erase;

  // inputs: keys, queries and V^T (zero past the chunk's end), beta, and the
  // decay rates of this thread's row and token segment in registers
  constexpr int V8 = DK / 8;
  const int ri = t % DK, sg = t / DK;
  float sv[SEGL];
#pragma unroll
  for (int u = 0; u < SEGL; ++u) {
    const int j = sg * SEGL + u;
    sv[u] = j < n ? (p.per_head ? p.s[th(j)] : p.s[th(j) * DK + ri]) : 0.f;
  }
  // every load is issued before the first LDS store, so that the round
  // trips overlap
  constexpr int NE = CT * V8 / NTP;   // 16-byte vectors per thread and array
  static_assert(CT * V8 % NTP == 0, "whole vectors per thread");
  uint4 kv[NE], qv[NE], vv[NE];
#pragma unroll
  for (int r = 0; r < NE; ++r) {
    const int e = t + r * NTP;
    const int j = e / V8, g = e % V8;
    const int jv = e % CT, gv = e / CT;   // V^T: consecutive lanes, consecutive tokens
    kv[r] = qv[r] = vv[r] = make_uint4(0u, 0u, 0u, 0u);
    if (j < n) {
      kv[r] = ((const uint4*)p.k)[th(j) * V8 + g];
      qv[r] = ((const uint4*)p.q)[th(j) * V8 + g];
    }
    if (jv < n) vv[r] = ((const uint4*)p.v)[th(jv) * V8 + gv];
  }
  const float bt = t < CT && t < n ? p.beta[th(t)] : 0.f;
#pragma unroll
  for (int r = 0; r < NE; ++r) {
    const int e = t + r * NTP;
    const int j = e / V8, g = e % V8;
    const int jv = e % CT, gv = e / CT;
    *(uint4*)&sm.k[j][8 * g] = kv[r];
    *(uint4*)&sm.q[j][8 * g] = qv[r];
    const uint32_t x[4] = {vv[r].x, vv[r].y, vv[r].z, vv[r].w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      sm.vt[8 * gv + 2 * u][jv] = (uint16_t)(x[u] & 0xFFFFu);
      sm.vt[8 * gv + 2 * u + 1][jv] = (uint16_t)(x[u] >> 16);
    }
  }
  if (t < CT) sm.beta[t] = bt;
  __syncthreads();

  // decay scan and EMA sums over this thread's segment (token order, double)
  {
    float cs = 0.f;
    double qm = 0.0, qe = 0.0;
#pragma unroll
    for (int u = 0; u < SEGL; ++u) {
      const int j = sg * SEGL + u;
      cs += sv[u];
      sm.u0.c[j][ri] = cs;
      if (j < n) {
        const double z = decay_sample(sv[u]);
        const double y = erase ? erase_sample(bf16_f32(sm.k[j][ri]), sm.beta[j]) : 0.0;
        if (j == 0) {
          sm.u1.seg.first[0][ri] = z;
          sm.u1.seg.first[1][ri] = y;
        }
        qm = p.one_minus_alpha * qm + p.alpha * z;
        qe = p.one_minus_alpha * qe + p.alpha * y;
      }
    }
    sm.u1.seg.csum[sg][ri] = cs;
    sm.u1.seg.em[sg][0][ri] = qm;
    sm.u1.seg.em[sg][1][ri] = qe;
  }
  __syncthreads();
  {
    // later segments start from the sum of the earlier ones
    float off = 0.f;
    for (int s2 = 0; s2 < sg; ++s2) off += sm.u1.seg.csum[s2][ri];
    if (sg > 0) {
#pragma unroll
      for (int u = 0; u < SEGL; ++u) sm.u0.c[sg * SEGL + u][ri] += off;
    }
    if (sg == 0) {
      // EMA over the chunk: segment sums combined in token order
      double qm = sm.u1.seg.em[0][0][ri], qe = sm.u1.seg.em[0][1][ri];
      for (int s2 = 1; s2 < SEGS; ++s2) {
        const int nv = min(max(n - s2 * SEGL, 0), SEGL);
        double P = 1.0;
        for (int u = 0; u < nv; ++u) P *= p.one_minus_alpha;
        qm = P * qm + sm.u1.seg.em[s2][0][ri];
        qe = P * qe + sm.u1.seg.em[s2][1][ri];
      }
      double* ema = (double*)(out + CW::ema);
      ema[ri] = qm;
      ema[DK + ri] = qe;
      ema[2 * DK + ri] = sm.u1.seg.first[0][ri];
      ema[3 * DK + ri] = sm.u1.seg.first[1][ri];
    }
  }
  __syncthreads();

  // Qhat (row-major), Khat^T (LDS), Ktil^T and gamma_{n-1}, hi and lo
  // planes; decay factors with the correctly rounded float32 exponential
  {
    uint16_t* qh = (uint16_t*)(out + CW::qh);
    for (int e = t; e < CT * V8; e += NTP) {
      const int j = e / V8, i0 = 8 * (e % V8);
      const uint4 qv = *(const uint4*)&sm.q[j][i0];
      const float4 c0 = *(const float4*)&sm.u0.c[j][i0], c1 = *(const float4*)&sm.u0.c[j][i0 + 4];
      const float cc[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
      const uint32_t qw[4] = {qv.x, qv.y, qv.z, qv.w};
      uint32_t oh[4], ol[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        split2(bf16_f32((uint16_t)(qw[u] & 0xFFFFu)) * expf(-cc[2 * u]),
               bf16_f32((uint16_t)(qw[u] >> 16)) * expf(-cc[2 * u + 1]), oh[u], ol[u]);
      *(uint4*)&qh[j * DK + i0] = make_uint4(oh[0], oh[1], oh[2], oh[3]);
      *(uint4*)&qh[CT * DK + j * DK + i0] = make_uint4(ol[0], ol[1], ol[2], ol[3]);
    }
    uint16_t* ktt = (uint16_t*)(out + CW::ktt);
    for (int e = t; e < CT * DK; e += NTP) {
      const int i = e / CT, j = e % CT;
      const float c = sm.u0.c[j][i], ce = sm.u0.c[CT - 1][i];
      const float kk = bf16_f32(sm.k[j][i]);
      const float kh = kk * expf(-c), kt = kk * expf(c - ce);
      const uint16_t hh = bf16_rne(kh), th = bf16_rne(kt);
      sm.kht[0][i][j] = hh;
      sm.kht[1][i][j] = bf16_lo(kh, hh);
      ktt[e] = th;
      ktt[CT * DK + e] = bf16_lo(kt, th);
    }
    if (t < DK) ((float*)(out + CW::gend))[t] = (float)exp(-(double)sm.u0.c[CT - 1][t]);
  }

  // L (LDS) and A (global, bf16), block row J = w % 4: tiles (J, T <= J)
  // of parity w / 4
  {
    uint16_t* am = (uint16_t*)(out + CW::am);
    const int J = w & 3, par = w >> 2;
    const int k8 = 8 * (lane >> 4);
    const int jr = 16 * J + (lane & 15);
    bool wide = false;
    for (int i = lane; i < DK; i += WAVE) {
      const float cr = J ? sm.u0.c[16 * J - 1][i] : 0.f;
      wide = wide || (sm.u0.c[16 * J + 15][i] - cr > SPLIT_SPAN);
    }
    const bool diag_valu = __ballot(wide) != 0;
    f32x4 accL[4], accA[4];
#pragma unroll
    for (int T = 0; T < 4; ++T) {
      accL[T] = f32x4{0.f, 0.f, 0.f, 0.f};
      accA[T] = accL[T];
    }
    for (int ks = 0; ks < DK / 32; ++ks) {
      const int i0 = 32 * ks + k8;
      float cr[8];
      if (J) {
        const float4 a0 = *(const float4*)&sm.u0.c[16 * J - 1][i0];
        const float4 a1 = *(const float4*)&sm.u0.c[16 * J - 1][i0 + 4];
        cr[0] = a0.x; cr[1] = a0.y; cr[2] = a0.z; cr[3] = a0.w;
        cr[4] = a1.x; cr[5] = a1.y; cr[6] = a1.z; cr[7] = a1.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) cr[e] = 0.f;
      }
      const float4 j0 = *(const float4*)&sm.u0.c[jr][i0], j1 = *(const float4*)&sm.u0.c[jr][i0 + 4];
      const float cj[8] = {j0.x, j0.y, j0.z, j0.w, j1.x, j1.y, j1.z, j1.w};
      const uint4 kv = *(const uint4*)&sm.k[jr][i0], qv = *(const uint4*)&sm.q[jr][i0];
      const uint32_t kw[4] = {kv.x, kv.y, kv.z, kv.w}, qw[4] = {qv.x, qv.y, qv.z, qv.w};
      uint32_t akh[4], akl[4], aqh[4], aql[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float f0 = expf(cr[2 * e] - cj[2 * e]), f1 = expf(cr[2 * e + 1] - cj[2 * e + 1]);
        split2(bf16_f32((uint16_t)(kw[e] & 0xFFFFu)) * f0, bf16_f32((uint16_t)(kw[e] >> 16)) * f1,
               akh[e], akl[e]);
        split2(bf16_f32((uint16_t)(qw[e] & 0xFFFFu)) * f0, bf16_f32((uint16_t)(qw[e] >> 16)) * f1,
               aqh[e], aql[e]);
      }
      const uint4 AKh = make_uint4(akh[0], akh[1], akh[2], akh[3]);
      const uint4 AKl = make_uint4(akl[0], akl[1], akl[2], akl[3]);
      const uint4 AQh = make_uint4(aqh[0], aqh[1], aqh[2], aqh[3]);
      const uint4 AQl = make_uint4(aql[0], aql[1], aql[2], aql[3]);
#pragma unroll
      for (int T = 0; T < 4; ++T) {
        if ((T & 1) != par || T > J || (T == J && diag_valu)) continue;
        const int jt = 16 * T + (lane & 15);
        const float4 t0 = *(const float4*)&sm.u0.c[jt][i0], t1 = *(const float4*)&sm.u0.c[jt][i0 + 4];
        const float ct[8] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
        const uint4 tv = *(const uint4*)&sm.k[jt][i0];
        const uint32_t tw[4] = {tv.x, tv.y, tv.z, tv.w};
        uint32_t bkh[4], bkl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          split2(bf16_f32((uint16_t)(tw[e] & 0xFFFFu)) * expf(ct[2 * e] - cr[2 * e]),
                 bf16_f32((uint16_t)(tw[e] >> 16)) * expf(ct[2 * e + 1] - cr[2 * e + 1]), bkh[e],
                 bkl[e]);
        const uint4 BKh = make_uint4(bkh[0], bkh[1], bkh[2], bkh[3]);
        const uint4 BKl = make_uint4(bkl[0], bkl[1], bkl[2], bkl[3]);
        if (erase) accL[T] = mma3(AKh, AKl, BKh, BKl, accL[T]);
        accA[T] = mma3(AQh, AQl, BKh, BKl, accA[T]);
      }
    }
#pragma unroll
    for (int T = 0; T < 4; ++T) {
      if ((T & 1) != par) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = 16 * J + 4 * (lane >> 4) + r, tau = 16 * T + (lane & 15);
        if (T > J) {
          sm.u1.L[j][tau] = 0.f;
          am[j * CT + tau] = 0;
          am[CT * CT + j * CT + tau] = 0;
        } else if (T < J || !diag_valu) {
          sm.u1.L[j][tau] = tau < j ? accL[T][r] : 0.f;
          const float a = tau <= j ? accA[T][r] : 0.f;
          const uint16_t ah = bf16_rne(a);
          am[j * CT + tau] = ah;
          am[CT * CT + j * CT + tau] = bf16_lo(a, ah);
        }
      }
    }
    if (diag_valu && (J & 1) == par) {
      // one exponential per pair and row: exp(c_tau - c_j) <= 1 for tau <= j
      for (int pr = lane; pr < 256; pr += WAVE) {
        const int j = 16 * J + pr / 16, tau = 16 * J + pr % 16;
        float l = 0.f, a = 0.f;
        if (tau <= j) {
          for (int i = 0; i < DK; ++i) {
            const float kt = bf16_f32(sm.k[tau][i]) * expf(sm.u0.c[tau][i] - sm.u0.c[j][i]);
            l = fmaf(bf16_f32(sm.k[j][i]), kt, l);
            a = fmaf(bf16_f32(sm.q[j][i]), kt, a);
          }
        }
        sm.u1.L[j][tau] = (tau < j && erase) ? l : 0.f;
        const float av = tau <= j ? a : 0.f;
        const uint16_t ah = bf16_rne(av);
        am[j * CT + tau] = ah;
        am[CT * CT + j * CT + tau] = bf16_lo(av, ah);
      }
    }
  }
  __syncthreads();

  // T = (I + N)^-1 with N = diag(beta) L, by 16-row blocks.  Diagonal
  // blocks: forward substitution, column m of block w on lane m.
  if (w < 4 && lane < 16) {
    const int J = w, m = lane;
    float Tc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int tau = 0; tau < j; ++tau) acc = fmaf(sm.u1.L[16 * J + j][16 * J + tau], Tc[tau], acc);
      Tc[j] = j == m ? 1.f : (j > m ? -sm.beta[16 * J + j] * acc : 0.f);
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) sm.u0.t.T[16 * J + j][16 * J + m] = Tc[j];
  }
  // off-diagonal blocks by distance d: T_JK = -T_JJ sum_{M=K}^{J-1} N_JM T_MK
  for (int d = 1; d < 4; ++d) {
    __syncthreads();
    const int J = w, K = w - d;
    const int a = lane / 4, b4 = 4 * (lane % 4);   // output row, four columns
    if (w < 4 && K >= 0) {
      float x[4] = {0.f, 0.f, 0.f, 0.f};
      for (int M = K; M < J; ++M) {
#pragma unroll
        for (int tau = 0; tau < 16; ++tau) {
          const float nv = sm.u1.L[16 * J + a][16 * M + tau];
          const float4 tv = *(const float4*)&sm.u0.t.T[16 * M + tau][16 * K + b4];
          x[0] = fmaf(nv, tv.x, x[0]);
          x[1] = fmaf(nv, tv.y, x[1]);
          x[2] = fmaf(nv, tv.z, x[2]);
          x[3] = fmaf(nv, tv.w, x[3]);
        }
      }
      const float bj = sm.beta[16 * J + a];
#pragma unroll
      for (int u = 0; u < 4; ++u) sm.u0.t.X[w][a][b4 + u] = bj * x[u];
    }
    __syncthreads();
    if (w < 4 && K >= 0) {
      float y[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int tau = 0; tau < 16; ++tau) {
        const float tv = sm.u0.t.T[16 * J + a][16 * J + tau];
        const float4 xv = *(const float4*)&sm.u0.t.X[w][tau][b4];
        y[0] = fmaf(tv, xv.x, y[0]);
        y[1] = fmaf(tv, xv.y, y[1]);
        y[2] = fmaf(tv, xv.z, y[2]);
        y[3] = fmaf(tv, xv.w, y[3]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) sm.u0.t.T[16 * J + a][16 * K + b4 + u] = -y[u];
    }
  }
  __syncthreads();
  for (int e = t; e < CT * CT; e += NTP) {
    const int j = e / CT, m = e % CT;
    const float x = m <= j ? sm.u0.t.T[j][m] * sm.beta[m] : 0.f;
    const uint16_t xh = bf16_rne(x);
    sm.tb[j][m] = xh;
    sm.u0.t.tbl[j][m] = bf16_lo(x, xh);
  }
  __syncthreads();

  // Uv = T diag(beta) V and Wk = T diag(beta) Khat: token tile w % 4,
  // column half w / 4
  {
    constexpr int NC = DK / 32;   // 16-column tiles per half
    const int J = w & 3, c0 = (w >> 2) * NC;
    const int k8 = 8 * (lane >> 4);
    f32x4 au[NC], aw[NC];
#pragma unroll
    for (int ct = 0; ct < NC; ++ct) {
      au[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
      aw[ct] = au[ct];
    }
#pragma unroll
    for (int ks = 0; ks < CT / 32; ++ks) {
      if (32 * ks > 16 * J + 15) break;   // T is lower triangular
      const uint4 ah = *(const uint4*)&sm.tb[16 * J + (lane & 15)][32 * ks + k8];
      const uint4 al = *(const uint4*)&sm.u0.t.tbl[16 * J + (lane & 15)][32 * ks + k8];
#pragma unroll
      for (int ct = 0; ct < NC; ++ct) {
        const uint4 bv = *(const uint4*)&sm.vt[16 * (c0 + ct) + (lane & 15)][32 * ks + k8];
        au[ct] = mma2(ah, al, bv, au[ct]);
        if (erase) {
          const uint4 bh = *(const uint4*)&sm.kht[0][16 * (c0 + ct) + (lane & 15)][32 * ks + k8];
          const uint4 bl = *(const uint4*)&sm.kht[1][16 * (c0 + ct) + (lane & 15)][32 * ks + k8];
          aw[ct] = mma3(ah, al, bh, bl, aw[ct]);
        }
      }
    }
    float* uv = (float*)(out + CW::uv);
    uint16_t* wk = (uint16_t*)(out + CW::wk);
#pragma unroll
    for (int ct = 0; ct < NC; ++ct) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = 16 * J + 4 * (lane >> 4) + r, i = 16 * (c0 + ct) + (lane & 15);
        uv[j * DK + i] = au[ct][r];
        const uint16_t wh = bf16_rne(aw[ct][r]);
        wk[j * DK + i] = wh;
        wk[CT * DK + j * DK + i] = bf16_lo(aw[ct][r], wh);
      }
    }
  }
}

// Units unit0 + blockIdx.x of a group.  Beside the per-interval kernels the
// group is prepared by a series of launches of a few blocks each, which
// leave compute units to the intervals running on the other stream.
template <int DK>
__global__ void __launch_bounds__(NTP) k_chunk_prep(KParams p, int C, uint8_t* cws, int unit0) {
  __shared__ PrepSmem<DK> sm;
  prep_unit<DK>(p, C, cws, unit0 + blockIdx.x, sm);
}

template <int DK>
struct ApplySmem {
  static constexpr int SS = DK + 8;
  static constexpr int US = CT + 8;
  uint16_t s0t[2][SLICE][SS];   // S0 of the slice, transposed, bf16 hi and lo planes
  uint16_t ut[2][SLICE][US];    // U of the slice, transposed, bf16 hi and lo planes
};

// The chunk record's operands one wave of the apply holds in registers:
// hi and lo planes of its token tile of Wk, Qhat and A, of its state-row
// tiles of Ktil^T, its rows of Uv in the slice and gamma_{n-1} of its rows.
template <int DK>
struct ApplyFrags {
  static constexpr int RT = DK / 64;   // 16-row state tiles per wave
  static constexpr int KS = DK / 32;   // k-steps over the state's rows
  uint4 fw[2][KS], fq[2][KS], fa[2][CT / 32], fk[2][RT][CT / 32];
  float fu[4][4], fg[RT][4];
};

// Wave w (of the four of a slice) of slice sl; `in` is the head's chunk record.
// Requested in the order the products use them (loads complete in order).
template <int DK>
__device__ __forceinline__ void load_frags(const uint8_t* in, int sl, int w, ApplyFrags<DK>& f) {
  using CW = ChunkWs<DK>;
  constexpr int RT = ApplyFrags<DK>::RT, KS = ApplyFrags<DK>::KS;
  const int lane = lane_id(), k8 = 8 * (lane >> 4), l16 = lane & 15;
  const int jrow = 16 * w + l16;
  const uint16_t* wk = (const uint16_t*)(in + CW::wk);
  const uint16_t* qh = (const uint16_t*)(in + CW::qh);
  const uint16_t* am = (const uint16_t*)(in + CW::am);
  const uint16_t* ktt = (const uint16_t*)(in + CW::ktt);
  const float* uv = (const float*)(in + CW::uv);
  const float* gend = (const float*)(in + CW::gend);
  constexpr int PL = CT * DK;            // elements of one plane
  // W = Wk S0 and O = Qhat S0
#pragma unroll
  for (int hl = 0; hl < 2; ++hl)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      f.fw[hl][ks] = *(const uint4*)&wk[hl * PL + jrow * DK + 32 * ks + k8];   // used if erase
      f.fq[hl][ks] = *(const uint4*)&qh[hl * PL + jrow * DK + 32 * ks + k8];
    }
  // U = Uv - W
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      f.fu[ct][r] = uv[(16 * w + 4 * (lane >> 4) + r) * DK + SLICE * sl + 16 * ct + l16];
  // O += A U (blocks used up to the tile's last token)
#pragma unroll
  for (int hl = 0; hl < 2; ++hl)
#pragma unroll
    for (int ks = 0; ks < CT / 32; ++ks)
      f.fa[hl][ks] = *(const uint4*)&am[hl * CT * CT + jrow * CT + 32 * ks + k8];
  // S = gamma S0 + Ktil^T U
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) f.fg[rt][r] = gend[16 * (RT * w + rt) + 4 * (lane >> 4) + r];
#pragma unroll
  for (int hl = 0; hl < 2; ++hl)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ks = 0; ks < CT / 32; ++ks)
        f.fk[hl][rt][ks] = *(const uint4*)&ktt[hl * PL + (16 * (RT * w + rt) + l16) * CT + 32 * ks + k8];
}

// One write-back interval of one 64-column slice of one head, tokens
// [p.tok0, p.tok0 + p.ntk), by the four waves w of the slice (t: thread
// within them); every thread of the block calls it (two barriers).  s0(i, c)
// is the dequantised state at row i, column c of the slice.
// Writes the outputs, the float32 state, its per-slice row maxima and (slice
// 0) Gamma and the rate codes, as the token-sequential stats kernel does.
// Every product takes its operands as hi and lo bf16 planes (mma3), float32
// accumulation.
template <int DK, typename S0>
__device__ __forceinline__ void apply_slice(const KParams& p, const uint8_t* in, int bh, int sl, int w,
                                            int t, const ApplyFrags<DK>& f, ApplySmem<DK>& sm,
                                            S0 s0, float* rmax_lds = nullptr,
                                            double* gam_lds = nullptr) {
  using CW = ChunkWs<DK>;
  constexpr int RT = ApplyFrags<DK>::RT, KS = ApplyFrags<DK>::KS;
  const int nsl = p.dv / SLICE;
  const int b = bh / p.H, h = bh % p.H;
  const int lane = lane_id();
  const int n = p.ntk;
  const int k8 = 8 * (lane >> 4), l16 = lane & 15;
  const bool erase = !p.no_erase;

  // S0^T in LDS as hi and lo planes for the products (this lane's state-tile
  // positions; the accumulator of S_n is formed from S0 again further down,
  // so that it is not held through the first products)
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * (RT * w + rt) + 4 * (lane >> 4) + r;
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        const int c = 16 * ct + l16;
        const float x = s0(i, c);
        const uint16_t xh = bf16_rne(x);
        sm.s0t[0][c][i] = xh;
        sm.s0t[1][c][i] = bf16_lo(x, xh);
      }
    }
  }
  __syncthreads();

  // W = Wk S0 and O = Qhat S0 for token tile w
  f32x4 aw[4], ao[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    aw[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    ao[ct] = aw[ct];
  }
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const uint4 bh_ = *(const uint4*)&sm.s0t[0][16 * ct + l16][32 * ks + k8];
      const uint4 bl_ = *(const uint4*)&sm.s0t[1][16 * ct + l16][32 * ks + k8];
      if (erase) aw[ct] = mma3(f.fw[0][ks], f.fw[1][ks], bh_, bl_, aw[ct]);
      ao[ct] = mma3(f.fq[0][ks], f.fq[1][ks], bh_, bl_, ao[ct]);
    }
  }
  // U = Uv - W, transposed into LDS as hi and lo planes
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = 16 * w + 4 * (lane >> 4) + r, c = 16 * ct + l16;
      const float u = f.fu[ct][r] - aw[ct][r];
      const uint16_t uh = bf16_rne(u);
      sm.ut[0][c][j] = uh;
      sm.ut[1][c][j] = bf16_lo(u, uh);
    }
  }
  __syncthreads();

  // O += A U (A is lower triangular: k-steps up to the tile's last token)
#pragma unroll
  for (int ks = 0; ks < CT / 32; ++ks) {
    if (32 * ks > 16 * w + 15) break;
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const uint4 uh = *(const uint4*)&sm.ut[0][16 * ct + l16][32 * ks + k8];
      const uint4 ul = *(const uint4*)&sm.ut[1][16 * ct + l16][32 * ks + k8];
      ao[ct] = mma3(f.fa[0][ks], f.fa[1][ks], uh, ul, ao[ct]);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int j = 16 * w + 4 * (lane >> 4) + r;
    if (j < n) {
      float* orow = p.o + (((size_t)b * p.T + p.tok0 + j) * p.H + h) * p.dv + SLICE * sl;
#pragma unroll
      // outputs and state are read by other kernels only: nontemporal
      // stores keep them from filling the L2 that the next kernel's
      // start must write back
      for (int ct = 0; ct < 4; ++ct) __builtin_nontemporal_store(ao[ct][r], &orow[16 * ct + l16]);
    }
  }

  // S_n = gamma_{n-1} * S0 + Ktil^T U (float32 gamma_{n-1} * S0 at this
  // lane's state-tile positions as the accumulator)
  f32x4 acc[RT][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
        acc[rt][ct][r] = f.fg[rt][r] * s0(16 * (RT * w + rt) + 4 * (lane >> 4) + r, 16 * ct + l16);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int ks = 0; ks < CT / 32; ++ks) {
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        const uint4 uh = *(const uint4*)&sm.ut[0][16 * ct + l16][32 * ks + k8];
        const uint4 ul = *(const uint4*)&sm.ut[1][16 * ct + l16][32 * ks + k8];
        acc[rt][ct] = mma3(f.fk[0][rt][ks], f.fk[1][rt][ks], uh, ul, acc[rt][ct]);
      }
    }
  }
  // float32 state and per-slice row maxima
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * (RT * w + rt) + 4 * (lane >> 4) + r;
      float* srow = p.ws_s32 + ((size_t)bh * DK + i) * p.dv + SLICE * sl;
      float m = 0.f;
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        const float x = acc[rt][ct][r];
        __builtin_nontemporal_store(x, &srow[16 * ct + l16]);
        m = fmaxf(m, fabsf(x));
      }
      m = max16(m);
      if (l16 == 0) {
        p.ws_rpart[((size_t)bh * DK + i) * nsl + sl] = m;
        if (rmax_lds != nullptr) rmax_lds[sl * DK + i] = m;
      }
    }
  }
  if (sl == 0 && t < DK) {
    // Gamma and the rate codes after the chunk (k_chunk_rates)
    const double gm = ((const double*)(in + CW::gam))[t];
    p.ws_gam[(size_t)bh * DK + t] = gm;
    if (gam_lds != nullptr) gam_lds[t] = gm;
    p.ws_zr[(size_t)bh * DK + t] = ((const uint32_t*)(in + CW::zr))[t];
  }
}

// One write-back interval of one 64-column slice of one head from the
// record's state (block = (head, slice), see slice_block).
template <int DK>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2)))
    k_chunk_apply(KParams p, const uint8_t* cw) {
  using CW = ChunkWs<DK>;
  const int nsl = p.dv / SLICE;
  int bh, sl;
  slice_block(p.B * p.H, nsl, bh, sl);
  const int t = threadIdx.x, w = t / WAVE;
  const uint8_t* in = cw + (size_t)bh * CW::bytes;
  const Layout L = p.L;
  const uint8_t* rec = slot_ptr(p.records, L.slot, bh);
  __shared__ MetaSmem<DK> meta;
  __shared__ ApplySmem<DK> sm;
  extern __shared__ uint4 dyn_lds[];
  uint32_t* words = (uint32_t*)dyn_lds;

  // The state record's metadata and the slice's code words are requested
  // first and every operand of the products after them (loads complete in
  // order: the dequantisation waits for the record only).  Code words: word
  // kw of column sl*64 + c at words[kw*64 + c]; at most d_k MAX_B / 32 words
  // per column.
  const MetaFetch mf = meta_fetch<DK>(rec, L);
  constexpr int Q = SLICE / 4, WMAX = ((DK * MAX_B / 32) * Q + NT - 1) / NT;
  const u32x4* src = (const u32x4*)(rec + L.codes_off);
  const int n4 = L.wc * Q;
  u32x4 wv[WMAX];
#pragma unroll
  for (int q = 0; q < WMAX; ++q) {
    // indices past the last word read and store the last word again (the
    // same value as its owner): no branch, so the loads stay up here
    const int e = min(t + q * NT, n4 - 1);
    wv[q] = src[(size_t)(e / Q) * (p.dv / 4) + sl * Q + e % Q];
  }
  ApplyFrags<DK> f;
  load_frags<DK>(in, sl, w, f);
#pragma unroll
  for (int q = 0; q < WMAX; ++q) ((u32x4*)words)[min(t + q * NT, n4 - 1)] = wv[q];
  meta_form<DK, SLICE>(mf, p.bmax, meta);   // its barrier covers the staging
  auto s0 = [&](int i, int c) {
    const uint4 d = meta.desc[i];
    const int sh = (int)(d.y & 31u), bw = (int)(d.y >> 8);
    const float mul = __builtin_bit_cast(float, d.z), add = __builtin_bit_cast(float, d.w);
    const uint32_t lo = words[d.x + c], hi = words[d.x + SLICE + c];
    const int code = __builtin_amdgcn_sbfe((int)__builtin_amdgcn_alignbit(hi, lo, (uint32_t)sh), 0, bw);
    return ((float)code + add) * mul;
  };
  apply_slice<DK>(p, in, bh, sl, w, t, f, sm, s0);
}

// The same interval for all slices of one head in one block (four waves per
// slice, block = head), used when the normalisation groups lie within a head:
// the block then holds every row's maximum and Gamma and forms the allocation
// weights itself (row maxima over the slices, group RMS, keys into ws_c), so
// that the allocation that follows only selects.
template <int DK>
__global__ void __launch_bounds__((DK / SLICE) * NT) __attribute__((amdgpu_waves_per_eu(2)))
    k_chunk_apply_head(KParams p, const uint8_t* cw) {
  using CW = ChunkWs<DK>;
  constexpr int NSL = DK / SLICE;
  const int bh = blockIdx.x;
  const int t = threadIdx.x, sl = t / NT, tl = t % NT, w = tl / WAVE;
  const uint8_t* in = cw + (size_t)bh * CW::bytes;
  const Layout L = p.L;
  const uint8_t* rec = slot_ptr(p.records, L.slot, bh);
  __shared__ MetaSmem<DK> meta;
  __shared__ ApplySmem<DK> sm[NSL];
  __shared__ __align__(16) StatSmem<DK> st;
  __shared__ float rmax[NSL * DK];
  extern __shared__ uint4 dyn_lds[];
  uint32_t* words = (uint32_t*)dyn_lds;

  // The state record's metadata and code words are requested first and every
  // operand of the products after them: loads complete in order, so the
  // dequantisation below waits for the record only, with the operands still
  // in flight.  Code words: word kw of column j at words[kw d_v + j]; at most
  // d_k MAX_B / 32 words per column (wc <= that for every width bound).
  const MetaFetch mf = meta_fetch<DK>(rec, L);
  constexpr int NTH = NSL * NT, WMAX = ((DK * MAX_B / 32) * (DK / 4) + NTH - 1) / NTH;
  const u32x4* src = (const u32x4*)(rec + L.codes_off);
  const int n4 = L.wc * (DK / 4);
  u32x4 wv[WMAX];
#pragma unroll
  for (int q = 0; q < WMAX; ++q)
    wv[q] = src[min(t + q * NTH, n4 - 1)];   // past the end: the last word again, stored
                                              // where its owner stores it (no branch)
  ApplyFrags<DK> f;
  load_frags<DK>(in, sl, w, f);
#pragma unroll
  for (int q = 0; q < WMAX; ++q) ((u32x4*)words)[min(t + q * NTH, n4 - 1)] = wv[q];
  meta_form<DK, DK>(mf, p.bmax, meta);   // its barrier covers the staging
  auto s0 = [&](int i, int c) {
    const uint4 d = meta.desc[i];
    const int sh = (int)(d.y & 31u), bw = (int)(d.y >> 8);
    const float mul = __builtin_bit_cast(float, d.z), add = __builtin_bit_cast(float, d.w);
    const int j = SLICE * sl + c;
    const uint32_t lo = words[d.x + j], hi = words[d.x + DK + j];
    const int code = __builtin_amdgcn_sbfe((int)__builtin_amdgcn_alignbit(hi, lo, (uint32_t)sh), 0, bw);
    return ((float)code + add) * mul;
  };
  apply_slice<DK>(p, in, bh, sl, w, tl, f, sm[sl], s0, rmax, st.gam);
  __syncthreads();
  if (t < DK) {
    // the row's range: the maximum over the slices in slice order
    float m = rmax[t];
#pragma unroll
    for (int q = 1; q < NSL; ++q) m = fmaxf(m, rmax[q * DK + t]);
    st.R[t] = m;
  }
  __syncthreads();
  row_weights<DK>(p, bh, st, t);   // group RMS and keys into ws_c
}

// Rates of the chunks first_chunk .. first_chunk + nc - 1 (one group, records
// `cws`), one thread per row: the EMA over each chunk is m = (1 - alpha)^n m_0
// + Q (R24) with m_0 decoded from the rate codes the previous write-back
// stores; this chain depends on the inputs only (each write-back stores the
// codes of the EMA values, and the next interval continues from their decoded
// values), so it runs beside the intervals.  Writes each chunk's Gamma and
// rate codes into its record; `carry` holds every row's last codes for the
// next group (the call's first chunk starts from the record's codes, or from
// its first samples if the record is fresh).
template <int DK>
__global__ void __launch_bounds__(256) k_chunk_rates(KParams p, int C, uint8_t* cws, int first_chunk,
                                                     int nc, uint32_t* carry) {
  using CW = ChunkWs<DK>;
  const int nbh = p.B * p.H;
  const int gi = blockIdx.x * blockDim.x + threadIdx.x;
  if (gi >= nbh * DK) return;
  const int bh = gi / DK, t = gi % DK;
  bool fresh = false;
  uint32_t zr;
  if (first_chunk == 0) {
    const uint8_t* rec = slot_ptr(p.records, p.L.slot, bh);
    fresh = *(const unsigned*)rec == 0u;
    zr = (uint32_t)((const uint16_t*)(rec + p.L.z_off))[t] |
         ((uint32_t)((const uint16_t*)(rec + p.L.r_off))[t] << 16);
  } else {
    zr = carry[gi];
  }
  for (int c = 0; c < nc; ++c) {
    const int k = first_chunk + c;
    const int n = (p.T - k * C) < C ? (p.T - k * C) : C;
    uint8_t* out = cws + ((size_t)c * nbh + bh) * CW::bytes;
    const double* ema = (const double*)(out + CW::ema);
    double m0, e0;
    if (fresh) {
      m0 = ema[2 * DK + t];
      e0 = ema[3 * DK + t];
      fresh = false;
    } else {
      m0 = exp(-2.0 * logq_decode((uint16_t)(zr & 0xffffu)));
      e0 = 2.0 * (double)f16_to_f32((uint16_t)(zr >> 16));
    }
    double P = 1.0;
    for (int j = 0; j < n; ++j) P *= p.one_minus_alpha;
    const double m_run = P * m0 + ema[t];
    const double e_run = P * e0 + ema[DK + t];
    const double s_hat = -0.5 * log(m_run);
    const double r = 0.5 * e_run;
    ((double*)(out + CW::gam))[t] =
        p.gamma ? p.gamma[(size_t)bh * DK + t] : mode_gamma(p.weight_mode, s_hat, r, p.wb_C);
    zr = (uint32_t)logq_encode(s_hat) | ((uint32_t)r_encode(r) << 16);
    ((uint32_t*)(out + CW::zr))[t] = zr;
  }
  carry[gi] = zr;
}

size_t chunk_record_bytes(int dk) {
  return dk == 64 ? ChunkWs<64>::bytes : ChunkWs<128>::bytes;
}

int chunk_group(int nbh) {
  const int g = 4096 / nbh;
  return g < 1 ? 1 : (g > 16 ? 16 : g);
}

// Fork and join of the caller's auxiliary stream.  The preparation of the
// next group of chunks runs on `aux` while the current group's intervals run
// on `st` (the per-interval kernels fill only part of the chip).  The events
// that order the two streams are created by the call and destroyed when it
// returns; the library keeps no streams, events or locks of its own.  Once
// `aux` has been forked from `st`, every return path (errors included)
// records the end of the call's work on `aux` and makes `st` wait for it, so
// nothing of the call is left on `aux` after `st` -- in particular no branch
// of a graph being captured on `st` stays unjoined when the capture ends.
namespace {
struct AuxFork {
  hipStream_t st = nullptr, aux = nullptr;
  hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};   // fork, prep x2, join
  bool ok = false, forked = false;

  AuxFork(hipStream_t s, hipStream_t a) : st(s), aux(a) {
    if (aux == nullptr || aux == st) return;
    ok = true;
    for (int i = 0; i < 4 && ok; ++i)
      ok = hipEventCreateWithFlags(&ev[i], hipEventDisableTiming) == hipSuccess;
  }
  // aux waits for everything enqueued on st so far
  hipError_t fork() {
    hipError_t e = hipEventRecord(ev[0], st);
    if (e == hipSuccess) e = hipStreamWaitEvent(aux, ev[0], 0);
    if (e == hipSuccess) forked = true;
    return e;
  }
  ~AuxFork() {
    if (forked && hipEventRecord(ev[3], aux) == hipSuccess) (void)hipStreamWaitEvent(st, ev[3], 0);
    for (int i = 0; i < 4; ++i)
      if (ev[i] != nullptr) (void)hipEventDestroy(ev[i]);
  }
};
}  // namespace

// Blocks per preparation launch beside the intervals (one block fills a
// compute unit: its LDS and registers).
constexpr int PREP_SIDE_GRID = 128;

// Chunks per group.  With a side stream the groups grow from one chunk by
// about a quarter per group (floor(1.25^g): 1, 1, 1, 1, 2, 3, 3, 4, 5, 7, 9,
// ... up to gc), so that the first interval starts after one chunk's
// preparation and each later group's preparation (a chunk's takes about
// four fifths of an interval beside them) keeps pace with the previous
// group's intervals; without one, groups of gc chunks.  Once a size reaches
// gc every later one is gc.
static int group_size(int g, int gc, bool grow) {
  if (!grow) return gc;
  double a = 1.0;
  for (int j = 0; j < g && a < gc; ++j) a *= 1.25;
  const int n = (int)a;
  return n < gc ? n : gc;
}
static int group_first(int g, int gc, bool grow) {
  int c0 = 0;
  for (int i = 0; i < g; ++i) {
    const int k = group_size(i, gc, grow);
    c0 += k;
    if (k == gc) return c0 + (g - 1 - i) * gc;
  }
  return c0;
}

template <int DK>
static hipError_t run_chunked(KParams p, int C, hipStream_t st, hipStream_t aux_stream) {
  const int nbh = p.B * p.H, nsl = p.dv / SLICE;
  const int nch = (p.T + C - 1) / C;
  const int gc = chunk_group(nbh);
  const size_t dyn = (size_t)(p.L.wc + 1) * SLICE * 4;
  // groups within a head: one apply block per head forms the allocation keys
  const bool keys = p.G <= DK;
  const size_t dyn_head = (size_t)(p.L.wc + 1) * DK * 4;
  const size_t half = (size_t)gc * nbh * ChunkWs<DK>::bytes;   // records of up to gc chunks
  AuxFork fk(st, nch > 1 ? aux_stream : nullptr);
  const bool two = fk.ok;
  const bool grow = two;
  auto first = [&](int g) { return group_first(g, gc, grow); };
  auto count = [&](int g) {   // at most gc: one half of the records
    const int k = group_size(g, gc, grow), left = nch - first(g);
    return k < left ? k : left;
  };
  int ngr = 0;
  while (first(ngr) < nch) ++ngr;
  auto buf = [&](int g) { return p.ws_chunk + (two ? (size_t)(g & 1) * half : 0); };
  auto prep = [&](int g, hipStream_t s, bool side) {
    KParams q = p;
    q.tok0 = first(g) * C;
    const int units = nbh * count(g);
    const int step = side ? PREP_SIDE_GRID : units;
    for (int u0 = 0; u0 < units; u0 += step) {
      const hipError_t e = launch("prep", k_chunk_prep<DK>, units - u0 < step ? units - u0 : step,
                                  NTP, 0, s, q, C, buf(g), u0);
      if (e != hipSuccess) return e;
    }
    // the group's rates, continued from the previous group's (the decode
    // step's token-vector space of the workspace carries them between groups)
    return launch("rates", k_chunk_rates<DK>, (nbh * DK + 255) / 256, 256, 0, s, p, C, buf(g), first(g),
                  count(g), (uint32_t*)p.ws_hv);
  };
  auto group_of = [&](int k) {
    int g = 0;
    while (first(g + 1) <= k) ++g;
    return g;
  };
  auto rec = [&](int k) {   // chunk k's records
    const int g = group_of(k);
    return (const uint8_t*)(buf(g) + (size_t)(k - first(g)) * nbh * ChunkWs<DK>::bytes);
  };
  auto tokens = [&](int k) { return (p.T - k * C) < C ? (p.T - k * C) : C; };
  // A group prepared beside the intervals is enqueued a few launches at a
  // time, spread over the previous group's intervals: a queue holding many
  // launches of whole-compute-unit blocks held up the intervals' launches on
  // the main stream.  Its rates and its ready event follow its last launch.
  int pend_g = -1, pend_u0 = 0, pend_per = 1;
  auto feed = [&](int launches) -> hipError_t {
    if (pend_g < 0) return hipSuccess;
    KParams q = p;
    q.tok0 = first(pend_g) * C;
    const int units = nbh * count(pend_g);
    for (int i = 0; i < launches && pend_u0 < units; ++i, pend_u0 += PREP_SIDE_GRID) {
      const hipError_t e = launch("prep", k_chunk_prep<DK>,
                                  units - pend_u0 < PREP_SIDE_GRID ? units - pend_u0 : PREP_SIDE_GRID, NTP, 0,
                                  fk.aux, q, C, buf(pend_g), pend_u0);
      if (e != hipSuccess) return e;
    }
    if (pend_u0 < units) return hipSuccess;
    hipError_t e = launch("rates", k_chunk_rates<DK>, (nbh * DK + 255) / 256, 256, 0, fk.aux, p, C,
                          buf(pend_g), first(pend_g), count(pend_g), (uint32_t*)p.ws_hv);
    if (e == hipSuccess) e = hipEventRecord(fk.ev[1 + (pend_g & 1)], fk.aux);
    pend_g = -1;
    return e;
  };
  hipError_t e = prep(0, st, false);
  if (e != hipSuccess) return e;
  if (two && ngr > 1) {
    // group 1 is prepared beside group 0's intervals
    if ((e = fk.fork()) != hipSuccess) return e;
    if ((e = prep(1, fk.aux, true)) != hipSuccess) return e;
    if ((e = hipEventRecord(fk.ev[2], fk.aux)) != hipSuccess) return e;
  }
  // interval k: apply, allocation, requantisation
  for (int k = 0; k < nch; ++k) {
    const int g = group_of(k);
    if (k > 0 && k == first(g)) {
      if (two) {
        if (pend_g == g && (e = feed(0x7fffffff)) != hipSuccess) return e;   // all of it enqueued
        if ((e = hipStreamWaitEvent(st, fk.ev[1 + (g & 1)], 0)) != hipSuccess) return e;
      } else if ((e = prep(g, st, false)) != hipSuccess) {
        return e;
      }
    }
    p.tok0 = k * C;
    p.ntk = tokens(k);
    e = keys ? launch("apply", k_chunk_apply_head<DK>, nbh, nsl * NT, dyn_head, st, p, rec(k))
             : launch("apply", k_chunk_apply<DK>, nbh * nsl, NT, dyn, st, p, rec(k));
    if (e != hipSuccess) return e;
    if (two && k == first(g) + count(g) - 1 && g + 2 < ngr) {
      // chunk k's apply is the last read of group g's records: group g + 2
      // reuses them, prepared during group g + 1's intervals
      if ((e = feed(0x7fffffff)) != hipSuccess) return e;   // group g + 1 complete first
      if ((e = fk.fork()) != hipSuccess) return e;
      pend_g = g + 2;
      pend_u0 = 0;
      const int launches = (nbh * count(g + 2) + PREP_SIDE_GRID - 1) / PREP_SIDE_GRID;
      pend_per = (launches + count(g + 1) - 1) / count(g + 1);
    }
    if ((e = launch_chunk_writeback(p, nsl, st, keys)) != hipSuccess) return e;
    if (two && (e = feed(pend_per)) != hipSuccess) return e;
  }
  return hipSuccess;   // fk joins aux into st
}

hipError_t launch_prefill_chunked(const KParams& p, int C, hipStream_t st, hipStream_t aux) {
  if (p.dk == 64) return run_chunked<64>(p, C, st, aux);
  return run_chunked<128>(p, C, st, aux);
}

}  // namespace kda
