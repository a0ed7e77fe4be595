// Column-layout recurrence shared by the kernels that keep a head's state
// in registers: wave w owns rows [32w, 32w + 32), lane l owns columns
// l + 64c.  One token of eq. rule (Sec. 2) with the float32 contract: decay,
// the row contraction u = S'^T k as a sequential fma chain per 32-row block
// combined across waves by halving, the write, and o = S^T q the same way.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kda_device.hpp"
#include "kda_kernels.hpp"
#include "kda_record.hpp"

namespace kda {

// Per-row scalars of one token for the recurrence.
template <int DK>
struct RowSmem {
  float2 ak[DK];   // {fl32(exp(-s)), k}: first pass of the recurrence
  float2 gq[DK];   // {fl32(beta * k), q}: second pass
};

// Inputs of row t for the rate statistics: decay rate, key, beta.
struct RowIn {
  float s, k, beta;
};

// Per-row scalars of token `tok` of head bh into LDS (threads t < DK); returns
// the row's own inputs for the rate statistics.
template <int DK, bool BF16>
__device__ __forceinline__ RowIn load_rows(RowSmem<DK>& rs, const KParams& p, int bh, int tok) {
  const int t = threadIdx.x;
  RowIn in = {0.f, 0.f, 0.f};
  if (t < DK) {
    const int b = bh / p.H, h = bh % p.H;
    const size_t th = ((size_t)b * p.T + tok) * p.H + h;       // (b, tok, h)
    in.s = p.per_head ? p.s[th] : p.s[th * DK + t];
    in.beta = p.beta[th];
    in.k = in_f32<BF16>(p.k, th * DK + t);
    rs.ak[t] = make_float2((float)exp(-(double)in.s), in.k);
    rs.gq[t] = make_float2(in.beta * in.k, in_f32<BF16>(p.q, th * DK + t));
  }
  return in;
}

// Row scalars reach the lanes by DPP row broadcasts folded into the
// arithmetic: lane l of wave w holds the scalars of rows 32w + l % 16 (block
// 0) and 32w + 16 + l % 16 (block 1), replicated in the four 16-lane rows,
// and row_newbcast:r hands lane r's value of each 16-lane row to all of its
// lanes as the first operand.  Sixteen rows per asm block; the leading s_nop
// covers a vector write of a broadcast source just before the block.
#define KDA_P1(r)                                                                   \
  "v_mul_f32_dpp %" #r ", %17, %" #r " row_newbcast:" #r                           \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"                                       \
  "v_fmac_f32_dpp %16, %18, %" #r " row_newbcast:" #r                              \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
#define KDA_P2(r)                                                                   \
  "v_fmac_f32_dpp %" #r ", %17, %19 row_newbcast:" #r                              \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"                                       \
  "v_fmac_f32_dpp %16, %18, %" #r " row_newbcast:" #r                              \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
#define KDA_X16(X, o, c)                                                             \
  "+v"(X[o + 0][c]), "+v"(X[o + 1][c]), "+v"(X[o + 2][c]), "+v"(X[o + 3][c]),       \
      "+v"(X[o + 4][c]), "+v"(X[o + 5][c]), "+v"(X[o + 6][c]), "+v"(X[o + 7][c]),   \
      "+v"(X[o + 8][c]), "+v"(X[o + 9][c]), "+v"(X[o + 10][c]), "+v"(X[o + 11][c]), \
      "+v"(X[o + 12][c]), "+v"(X[o + 13][c]), "+v"(X[o + 14][c]), "+v"(X[o + 15][c])

// First pass over rows O..O+15 of column C: X_r = a_r X_r; acc = fma(k_r, X_r, acc)
// in row order.
template <int O, int C, int CPL>
__device__ __forceinline__ void pass1_16(float (&X)[ROW_BLOCK][CPL], float& acc, float A, float K) {
  asm("s_nop 1\n" KDA_P1(0) KDA_P1(1) KDA_P1(2) KDA_P1(3) KDA_P1(4) KDA_P1(5) KDA_P1(6) KDA_P1(7)
      KDA_P1(8) KDA_P1(9) KDA_P1(10) KDA_P1(11) KDA_P1(12) KDA_P1(13) KDA_P1(14) KDA_P1(15)
      : KDA_X16(X, O, C), "+v"(acc)
      : "v"(A), "v"(K));
}

// Second pass over rows O..O+15 of column C: X_r = fma(g_r, w, X_r);
// acc = fma(q_r, X_r, acc).
template <int O, int C, int CPL>
__device__ __forceinline__ void pass2_16(float (&X)[ROW_BLOCK][CPL], float& acc, float G, float Q,
                                         float wv) {
  asm("s_nop 1\n" KDA_P2(0) KDA_P2(1) KDA_P2(2) KDA_P2(3) KDA_P2(4) KDA_P2(5) KDA_P2(6) KDA_P2(7)
      KDA_P2(8) KDA_P2(9) KDA_P2(10) KDA_P2(11) KDA_P2(12) KDA_P2(13) KDA_P2(14) KDA_P2(15)
      : KDA_X16(X, O, C), "+v"(acc)
      : "v"(G), "v"(Q), "v"(wv));
}

// Token j's second pass fused with token j + 1's first pass, over the 32 rows
// of a lane's single column: per row r, X_r = fma(g_r, w, X_r),
// accO = fma(q_r, X_r, accO), X_r = a'_r X_r, accU = fma(k'_r, X_r, accU),
// i.e. the operations of pass2 (token j) and then pass1 (token j + 1) on
// every element, each chain still in row order; the rows are skewed (step s
// runs the first operation of row s, the next two of row s - 1 and the last
// of row s - 2), so every operand was written four instructions earlier and
// the two chains fill each other's latency.  Rows 0..15 take the sources
// (G0, Q0, A0, K0) of the first 16-row DPP block, rows 16..31 (G1, ...) of
// the second; the second asm block finishes rows 14 and 15.
__device__ __forceinline__ void fused_pass(float (&X)[ROW_BLOCK][1], float& accO, float& accU, float G0,
                                           float Q0, float A0, float K0, float G1, float Q1, float A1,
                                           float K1, float wv) {
  asm("s_nop 1\n"
      "v_fmac_f32_dpp %0, %18, %22 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %1, %18, %22 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %0 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %0, %20, %0 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %2, %18, %22 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %1 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %1, %20, %1 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %0 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %3, %18, %22 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %2 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %2, %20, %2 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %1 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %4, %18, %22 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %3 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %3, %20, %3 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %2 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %5, %18, %22 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %4 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %4, %20, %4 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %3 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %6, %18, %22 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %5 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %5, %20, %5 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %4 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %7, %18, %22 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %6 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %6, %20, %6 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %5 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %8, %18, %22 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %7 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %7, %20, %7 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %6 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %9, %18, %22 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %8 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %8, %20, %8 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %7 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %10, %18, %22 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %9 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %9, %20, %9 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %8 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %11, %18, %22 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %10 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %10, %20, %10 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %9 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %12, %18, %22 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %11 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %11, %20, %11 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %10 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %13, %18, %22 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %12 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %12, %20, %12 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %11 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %14, %18, %22 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %13 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %13, %20, %13 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %12 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %15, %18, %22 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %19, %14 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %14, %20, %14 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %21, %13 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      : "+v"(X[0][0]), "+v"(X[1][0]), "+v"(X[2][0]), "+v"(X[3][0]), "+v"(X[4][0]), "+v"(X[5][0]), "+v"(X[6][0]), "+v"(X[7][0]), "+v"(X[8][0]), "+v"(X[9][0]), "+v"(X[10][0]), "+v"(X[11][0]), "+v"(X[12][0]), "+v"(X[13][0]), "+v"(X[14][0]), "+v"(X[15][0]),
        "+v"(accO), "+v"(accU)
      : "v"(G0), "v"(Q0), "v"(A0), "v"(K0), "v"(wv));
  asm("s_nop 1\n"
      "v_fmac_f32_dpp %2, %20, %27 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %24, %1 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %1, %25, %1 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %26, %0 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %3, %20, %27 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %2 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %2, %22, %2 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %26, %1 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %4, %20, %27 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %3 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %3, %22, %3 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %2 row_newbcast:0 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %5, %20, %27 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %4 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %4, %22, %4 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %3 row_newbcast:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %6, %20, %27 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %5 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %5, %22, %5 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %4 row_newbcast:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %7, %20, %27 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %6 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %6, %22, %6 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %5 row_newbcast:3 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %8, %20, %27 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %7 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %7, %22, %7 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %6 row_newbcast:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %9, %20, %27 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %8 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %8, %22, %8 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %7 row_newbcast:5 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %10, %20, %27 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %9 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %9, %22, %9 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %8 row_newbcast:6 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %11, %20, %27 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %10 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %10, %22, %10 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %9 row_newbcast:7 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %12, %20, %27 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %11 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %11, %22, %11 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %10 row_newbcast:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %13, %20, %27 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %12 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %12, %22, %12 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %11 row_newbcast:9 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %14, %20, %27 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %13 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %13, %22, %13 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %12 row_newbcast:10 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %15, %20, %27 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %14 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %14, %22, %14 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %13 row_newbcast:11 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %16, %20, %27 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %15 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %15, %22, %15 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %14 row_newbcast:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %17, %20, %27 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %16 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %16, %22, %16 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %15 row_newbcast:13 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %18, %21, %17 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_mul_f32_dpp %17, %22, %17 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %16 row_newbcast:14 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "v_fmac_f32_dpp %19, %23, %17 row_newbcast:15 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      : "+v"(X[14][0]), "+v"(X[15][0]), "+v"(X[16][0]), "+v"(X[17][0]), "+v"(X[18][0]), "+v"(X[19][0]), "+v"(X[20][0]), "+v"(X[21][0]), "+v"(X[22][0]), "+v"(X[23][0]), "+v"(X[24][0]), "+v"(X[25][0]), "+v"(X[26][0]), "+v"(X[27][0]), "+v"(X[28][0]), "+v"(X[29][0]), "+v"(X[30][0]), "+v"(X[31][0]),
        "+v"(accO), "+v"(accU)
      : "v"(G1), "v"(Q1), "v"(A1), "v"(K1), "v"(Q0), "v"(A0), "v"(K0), "v"(wv));
}

template <int DK, int DV>
struct RecSmem {
  float up[DK / ROW_BLOCK][DV];
  float op[DK / ROW_BLOCK][DV];
};

// Halving combine of the per-wave partials of column col.
template <int DK, int DV>
__device__ __forceinline__ float combine_col(const float (&P)[DK / ROW_BLOCK][DV], int col) {
  constexpr int NWV = DK / ROW_BLOCK;
  float v[NWV];
#pragma unroll
  for (int p = 0; p < NWV; ++p) v[p] = P[p][col];
#pragma unroll
  for (int Lh = NWV / 2; Lh >= 1; Lh >>= 1) {
#pragma unroll
    for (int p = 0; p < Lh; ++p) v[p] = v[p] + v[p + Lh];
  }
  return v[0];
}

// One token of the gated delta rule on column-layout registers (eq. rule,
// KDA erase/write): S' = a S; u = S'^T k; S = S' + (beta k)(v - u)^T;
// o = S^T q.  Writes o to o_out (if non-null).  All threads must call.
template <int DK, int DV, bool BF16>
__device__ __forceinline__ void recur_token(float (&X)[ROW_BLOCK][DV / WAVE], const RowSmem<DK>& rs,
                            RecSmem<DK, DV>& sm, const void* v, size_t v_off, float* o_out,
                            bool erase, float* w_out = nullptr) {
  constexpr int CPL = DV / WAVE;
  static_assert(CPL <= 4, "columns per lane");
  const int w = threadIdx.x / WAVE, lane = lane_id();
  // row scalars of rows 32w + lane % 16 and 32w + 16 + lane % 16 (DPP sources)
  const float2 ak0 = rs.ak[w * ROW_BLOCK + (lane & 15)], ak1 = rs.ak[w * ROW_BLOCK + 16 + (lane & 15)];
  const float2 gq0 = rs.gq[w * ROW_BLOCK + (lane & 15)], gq1 = rs.gq[w * ROW_BLOCK + 16 + (lane & 15)];
  float vin[CPL];   // this lane's columns of v, loaded before the row sweep
#pragma unroll
  for (int c = 0; c < CPL; ++c) vin[c] = in_f32<BF16>(v, v_off + lane + WAVE * c);
  float acc[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
  pass1_16<0, 0, CPL>(X, acc[0], ak0.x, ak0.y);
  pass1_16<16, 0, CPL>(X, acc[0], ak1.x, ak1.y);
  if constexpr (CPL > 1) {
    pass1_16<0, 1, CPL>(X, acc[1], ak0.x, ak0.y);
    pass1_16<16, 1, CPL>(X, acc[1], ak1.x, ak1.y);
  }
  if constexpr (CPL > 2) {
    pass1_16<0, 2, CPL>(X, acc[2], ak0.x, ak0.y);
    pass1_16<16, 2, CPL>(X, acc[2], ak1.x, ak1.y);
    pass1_16<0, 3, CPL>(X, acc[3], ak0.x, ak0.y);
    pass1_16<16, 3, CPL>(X, acc[3], ak1.x, ak1.y);
  }
#pragma unroll
  for (int c = 0; c < CPL; ++c) sm.up[w][lane + WAVE * c] = acc[c];
  __syncthreads();
  float wv[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int col = lane + WAVE * c;
    const float u = combine_col<DK, DV>(sm.up, col);
    wv[c] = erase ? vin[c] - u : vin[c];   // no erasure: w = v
    acc[c] = 0.f;
    if (w_out != nullptr && w == 0) w_out[col] = wv[c];
  }
  pass2_16<0, 0, CPL>(X, acc[0], gq0.x, gq0.y, wv[0]);
  pass2_16<16, 0, CPL>(X, acc[0], gq1.x, gq1.y, wv[0]);
  if constexpr (CPL > 1) {
    pass2_16<0, 1, CPL>(X, acc[1], gq0.x, gq0.y, wv[1]);
    pass2_16<16, 1, CPL>(X, acc[1], gq1.x, gq1.y, wv[1]);
  }
  if constexpr (CPL > 2) {
    pass2_16<0, 2, CPL>(X, acc[2], gq0.x, gq0.y, wv[2]);
    pass2_16<16, 2, CPL>(X, acc[2], gq1.x, gq1.y, wv[2]);
    pass2_16<0, 3, CPL>(X, acc[3], gq0.x, gq0.y, wv[3]);
    pass2_16<16, 3, CPL>(X, acc[3], gq1.x, gq1.y, wv[3]);
  }
#pragma unroll
  for (int c = 0; c < CPL; ++c) sm.op[w][lane + WAVE * c] = acc[c];
  __syncthreads();
  if (o_out != nullptr && w == 0) {
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int col = lane + WAVE * c;
      o_out[col] = combine_col<DK, DV>(sm.op, col);
    }
  }
}

}  // namespace kda
