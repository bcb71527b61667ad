// tile16.hpp -- register-resident lower-triangular C x C tiles on gfx950 MFMA.
//
// A C x C matrix is cut into 16 x 16 blocks; a lower block-triangular matrix
// keeps its NB (NB + 1) / 2 blocks (NB = C / 16) in VGPRs of one wave.  Each
// block lives in one of two fragment forms of the 16 x 16 MFMA family (lane
// l, g = l >> 4, c = l & 15, four values v = 0..3 per lane):
//
//   column form (P): lane (g, c) holds M[4g + v][c]  -- the accumulator
//                    layout of v_mfma_*_16x16*, and the B-operand layout;
//   row form    (Q): lane (g, c) holds M[c][4g + v]  -- the A-operand layout.
//
// An MFMA computes D = X * Y from X in row form and Y in column form and
// leaves D in column form.  Swapping the operands computes D^T = Y^T X^T from
// the same fragments, which leaves D in row form.  Both factors' k-slots
// are indexed identically (k = 4g + v of the 16-wide block), so chained
// products never leave registers; the only layout changes are "multiply by
// the identity" MFMAs.
//
// Structural zeros: a matrix whose entries are known to vanish outside the
// sub-diagonals lo <= i - j <= hi skips every block that cannot intersect
// that band (a block at block-subdiagonal m spans i - j in [16m-15, 16m+15]).
// Entries that vanish inside a computed block are exact zeros by
// construction, so skipping is exact (NaN/Inf inputs aside).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

__host__ __device__ constexpr int nlower(int NB) { return NB * (NB + 1) / 2; }
__host__ __device__ constexpr int bidx(int I, int J) { return I * (I + 1) / 2 + J; }

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int lane_g() { return (threadIdx.x & 63) >> 4; }
__device__ __forceinline__ int lane_c() { return threadIdx.x & 15; }

// Can a block at block-subdiagonal m hold entries with lo <= i - j <= hi?
__device__ __forceinline__ bool blk_nz(int m, int lo, int hi) {
  return (16 * m + 15 >= lo) && (16 * m - 15 <= hi);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// ---------------------------------------------------------------------------
// element coordinates of a lane's value v inside block (I, J)

// i - j of value v held by this lane, column form
__device__ __forceinline__ int dP(int I, int J, int v) {
  return 16 * (I - J) + 4 * lane_g() + v - lane_c();
}
// i - j of value v held by this lane, row form
__device__ __forceinline__ int dQ(int I, int J, int v) {
  return 16 * (I - J) + lane_c() - 4 * lane_g() - v;
}

// identity block in either form (the two coincide)
__device__ __forceinline__ f32x4 eye4() {
  const int g = lane_g(), c = lane_c();
  f32x4 r;
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (c == 4 * g + v) ? 1.f : 0.f;
  return r;
}

// ---------------------------------------------------------------------------
// bf16 fragments

__device__ __forceinline__ bf16x4 to_bf16(f32x4 x) {
  bf16x4 r;
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (__bf16)x[v];
  return r;
}
__device__ __forceinline__ f32x4 to_f32(bf16x4 x) {
  f32x4 r;
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (float)x[v];
  return r;
}
__device__ __forceinline__ bf16x4 zero_bf4() {
  bf16x4 r;
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (__bf16)0.f;
  return r;
}

__device__ __forceinline__ bf16x8 cat8(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// D += X Y over two k-blocks at once (v_mfma_f32_16x16x32_bf16).
// OUTQ = false: D in column form (A = X row form, B = Y column form).
// OUTQ = true : D in row form    (A = Y column form, B = X row form).
// A single k-block is the same instruction with a zero second half: every bf16
// product uses this one opcode.  Chaining a 16x16x16 bf16 MFMA onto a
// 16x16x32 accumulator (SrcC = the previous result) got no wait states from
// this toolchain and read a stale accumulator on gfx950, so the two opcodes
// are never mixed.
template <bool OUTQ>
__device__ __forceinline__ f32x4 mma2(bf16x4 x0, bf16x4 x1, bf16x4 y0, bf16x4 y1, f32x4 acc) {
  const bf16x8 xa = cat8(x0, x1), ya = cat8(y0, y1);
  if constexpr (OUTQ)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(ya, xa, acc, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa, ya, acc, 0, 0, 0);
}
template <bool OUTQ>
__device__ __forceinline__ f32x4 mma1(bf16x4 x, bf16x4 y, f32x4 acc) {
  return mma2<OUTQ>(x, zero_bf4(), y, zero_bf4(), acc);
}

// fp32: one 16-wide k-block as four 16x16x4 MFMAs; instruction v contracts
// over k = 4g + v of the block.
template <bool OUTQ>
__device__ __forceinline__ f32x4 mma1(f32x4 x, f32x4 y, f32x4 acc) {
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    if constexpr (OUTQ)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y[v], x[v], acc, 0, 0, 0);
    else
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(x[v], y[v], acc, 0, 0, 0);
  }
  return acc;
}

// ---------------------------------------------------------------------------
// Operand traits: F = bf16x4 (bf16 compute) or f32x4 (fp32 compute)

template <typename F> struct Op;

template <> struct Op<bf16x4> {
  static __device__ __forceinline__ bf16x4 from(f32x4 x) { return to_bf16(x); }
  static __device__ __forceinline__ f32x4 f32(bf16x4 x) { return to_f32(x); }
  static __device__ __forceinline__ bf16x4 zero() { return zero_bf4(); }
  template <bool OUTQ>
  static __device__ __forceinline__ f32x4 pair(bf16x4 x0, bf16x4 x1, bf16x4 y0, bf16x4 y1,
                                               f32x4 acc) {
    return mma2<OUTQ>(x0, x1, y0, y1, acc);
  }
  template <bool OUTQ>
  static __device__ __forceinline__ f32x4 one(bf16x4 x, bf16x4 y, f32x4 acc) {
    return mma1<OUTQ>(x, y, acc);
  }
};

template <> struct Op<f32x4> {
  static __device__ __forceinline__ f32x4 from(f32x4 x) { return x; }
  static __device__ __forceinline__ f32x4 f32(f32x4 x) { return x; }
  static __device__ __forceinline__ f32x4 zero() { return zero4(); }
  template <bool OUTQ>
  static __device__ __forceinline__ f32x4 pair(f32x4 x0, f32x4 x1, f32x4 y0, f32x4 y1,
                                               f32x4 acc) {
    acc = mma1<OUTQ>(x0, y0, acc);
    return mma1<OUTQ>(x1, y1, acc);
  }
  template <bool OUTQ>
  static __device__ __forceinline__ f32x4 one(f32x4 x, f32x4 y, f32x4 acc) {
    return mma1<OUTQ>(x, y, acc);
  }
};

// ---------------------------------------------------------------------------
// D = X * Y for lower block-triangular X (row form), Y (column form).
// X has entries only on sub-diagonals [xlo, xhi], Y on [ylo, yhi]; only the
// part of D on [olo, ohi] is wanted (other blocks are written as 0).  The
// bounds are wave-uniform, so every skip is a scalar branch.

template <int NB, bool OUTQ, typename F>
__device__ __forceinline__ void lower_mm(f32x4 (&D)[nlower(NB)], const F (&X)[nlower(NB)],
                                         int xlo, int xhi, const F (&Y)[nlower(NB)], int ylo,
                                         int yhi, int olo, int ohi) {
  const int dlo = max(xlo + ylo, olo), dhi = min(xhi + yhi, ohi);
#pragma unroll
  for (int I = 0; I < NB; ++I) {
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 acc = zero4();
      if (blk_nz(I - J, dlo, dhi)) {
#pragma unroll
        for (int K = J; K <= I; K += 2) {
          const bool a0 = blk_nz(I - K, xlo, xhi) && blk_nz(K - J, ylo, yhi);
          if (K + 1 <= I) {
            const bool a1 = blk_nz(I - K - 1, xlo, xhi) && blk_nz(K + 1 - J, ylo, yhi);
            if (a0 && a1)
              acc = Op<F>::template pair<OUTQ>(X[bidx(I, K)], X[bidx(I, K + 1)], Y[bidx(K, J)],
                                               Y[bidx(K + 1, J)], acc);
            else if (a0)
              acc = Op<F>::template one<OUTQ>(X[bidx(I, K)], Y[bidx(K, J)], acc);
            else if (a1)
              acc = Op<F>::template one<OUTQ>(X[bidx(I, K + 1)], Y[bidx(K + 1, J)], acc);
          } else if (a0) {
            acc = Op<F>::template one<OUTQ>(X[bidx(I, K)], Y[bidx(K, J)], acc);
          }
        }
      }
      D[bidx(I, J)] = acc;
    }
  }
}

// Layout change of a lower block-triangular matrix by an identity MFMA.
// to_row: column form -> row form (Z = I Z with a row-form result);
// to_col: row form -> column form (Z = Z I with a column-form result).
template <int NB, typename F>
__device__ __forceinline__ void to_row(f32x4 (&D)[nlower(NB)], const F (&Zc)[nlower(NB)], int lo,
                                       int hi) {
  const F id = Op<F>::from(eye4());
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      D[bidx(I, J)] = blk_nz(I - J, lo, hi)
                          ? Op<F>::template one<true>(id, Zc[bidx(I, J)], zero4())
                          : zero4();
}
template <int NB, typename F>
__device__ __forceinline__ void to_col(f32x4 (&D)[nlower(NB)], const F (&Zr)[nlower(NB)], int lo,
                                       int hi) {
  const F id = Op<F>::from(eye4());
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      D[bidx(I, J)] = blk_nz(I - J, lo, hi)
                          ? Op<F>::template one<false>(Zr[bidx(I, J)], id, zero4())
                          : zero4();
}

template <int NB, typename F>
__device__ __forceinline__ void cvt_all(F (&Y)[nlower(NB)], const f32x4 (&X)[nlower(NB)]) {
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) Y[b] = Op<F>::from(X[b]);
}

}  // namespace gdn
