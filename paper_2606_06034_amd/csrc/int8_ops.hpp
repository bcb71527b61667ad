// int8_ops.hpp -- the INT8 arithmetic of the integer inverse (Section 3.5,
// Appendix G of arXiv 2606.06034): 8-bit codes (|q| <= 127) on int8 quad
// fragments, exact int32 products and sums, quantisation by the scale rule
// of intq.hpp, and the I8Ops width the shared engine (int_engine of
// intq.hpp) runs on, plus the per-tile quantiser's exponent.  Used by
// int8.hip and by the layer forward's integer-inverse mode.
#pragma once

#include "intq.hpp"

namespace gdn {
namespace i8 {

using namespace iq;

constexpr int kQ = 127, kQB = 7;

// round-half-even(y / 2^s) for 1 <= s <= 30 and |y| < 2^30
__device__ __forceinline__ int rne_pos(int y, int s) {
  return (y + (1 << (s - 1)) - 1 + ((y >> s) & 1)) >> s;
}
// any s >= 0 (s >= 31 rounds every |y| < 2^30 to 0)
__device__ __forceinline__ int rne_sh(int y, int s) {
  if (s <= 0) return y;
  if (s >= 31) return 0;
  return rne_pos(y, s);
}

// The helpers below visit only the blocks that can meet a band [lo, hi] of
// sub-diagonals; every other block of their operand is exactly zero by the
// structure of the computation, so skipping it changes no result.

// every entry scaled by 2^-s (s > 0: rounded half to even; s < 0: exact)
template <int NB>
__device__ __forceinline__ void scale_all(AccI<NB>& D, int s, int lo, int hi) {
  if (s > 0) {  // one test for all blocks (s is wave-uniform)
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (blk_nz(I - J, lo, hi))
#pragma unroll
          for (int v = 0; v < 4; ++v) D.a[bidx(I, J)][v] = rne_pos(D.a[bidx(I, J)][v], s);
  } else {
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (blk_nz(I - J, lo, hi))
#pragma unroll
          for (int v = 0; v < 4; ++v) D.a[bidx(I, J)][v] <<= -s;
  }
}

// exact int32 values (|y| < 2^30) of exponent e_in to codes by the scale
// rule, in place; exponent and non-zero flag through refs
template <int NB>
__device__ __forceinline__ void requant(AccI<NB>& D, int lo, int hi, int e_in, int& e_out,
                                        bool& nz) {
  const int amax = amax_of(D, lo, hi);
  nz = amax > 0;
  if (!nz) {
    e_out = 0;
    return;
  }
  const int s = shift_canon<kQ, kQB>(amax);
  if (s != 0) scale_all(D, s, lo, hi);
  e_out = e_in + s;
}

// ---------------------------------------------------------------------------

// The INT8 width for the shared integer engine (int_engine of intq.hpp):
// quads, exact int32 products and sums.
template <int NB> struct I8Ops {
  using Row = RowQ<NB>;
  using Col = ColQ<NB>;
  using Prod = AccI<NB>;
  static constexpr int kQ = i8::kQ;
  static constexpr int kQB = i8::kQB;                                 // |code| < 2^7
  static constexpr int kAccB = 14 + (NB == 1 ? 4 : NB == 2 ? 5 : 6);  // |product| < C 2^14
  static __device__ __forceinline__ void to_row(Row& X, const AccI<NB>& D, int lo, int hi) {
    to_rowq(X, D, lo, hi);
  }
  static __device__ __forceinline__ void to_col(Col& Y, const AccI<NB>& D, int lo, int hi) {
    to_colq(Y, D, lo, hi);
  }
  // the codes of the blocks of X that can meet [lo, hi] (others 0)
  static __device__ __forceinline__ void codes(AccI<NB>& D, const Row& X, int lo, int hi) {
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        D.a[bidx(I, J)] = blk_nz(I - J, lo, hi) ? unpack4(X.r[I].v[J]) : zero_i4();
  }
  template <bool OUTQ>
  static __device__ __forceinline__ void mm(Prod& D, const Row& X, const Col& Y, int lo, int hi) {
    mmi<NB, OUTQ>(D, X, Y, lo, hi);
  }
  // a product (exact int32) to codes
  static __device__ __forceinline__ void requant(Prod& D, AccI<NB>& q, int lo, int hi, int e_in,
                                                 int& e_out, bool& nz) {
    i8::requant(D, lo, hi, e_in, e_out, nz);
    q = D;
  }
  // codes to the finest scale that holds them (exact)
  static __device__ __forceinline__ void canon(AccI<NB>& q, int lo, int hi, int& e, bool& nz) {
    i8::requant(q, lo, hi, e, e, nz);
  }
  // X = q(X 2^eX + ys Y 2^eY) over [lo, hi] (X's band [xlo, hi], Y's
  // [ylo, hi]); Y is at the finest scale that holds it, and so is X when
  // xc.  Two terms with exponents 2 QB + 3 or more apart: the finer is below
  // an eighth of the output quantum and leaves the coarser's codes as they
  // are (at their finest scale); otherwise the sum is exact in int32 (below
  // 2^24).
  static __device__ __forceinline__ void add(AccI<NB>& X, int& eX, bool& nzX, int xlo, bool xc,
                                             const AccI<NB>& Y, int eY, bool nzY, int ys, int ylo,
                                             int lo, int hi) {
    const int g = !nzY ? 64 : nzX ? eX - eY : -64;
    if (g >= 2 * kQB + 3) {
      if (!xc) canon(X, xlo, hi, eX, nzX);
      return;
    }
    if (g <= -(2 * kQB + 3)) {
#pragma unroll
      for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int J = 0; J <= I; ++J)
          if (blk_nz(I - J, lo, hi))
            X.a[bidx(I, J)] = blk_nz(I - J, ylo, hi) ? Y.a[bidx(I, J)] * ys : zero_i4();
      eX = eY;
      nzX = true;
      return;
    }
    const int gx = max(g, 0), gy = max(-g, 0);
    const int e0 = min(eX, eY);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (blk_nz(I - J, lo, hi)) {
          i32x4 x = blk_nz(I - J, xlo, hi) ? X.a[bidx(I, J)] : zero_i4();
          const i32x4 y = blk_nz(I - J, ylo, hi) ? Y.a[bidx(I, J)] : zero_i4();
#pragma unroll
          for (int v = 0; v < 4; ++v) x[v] = (x[v] << gx) + ys * (y[v] << gy);
          X.a[bidx(I, J)] = x;
        }
    i8::requant(X, lo, hi, e0, eX, nzX);
  }
  static __device__ __forceinline__ void row_to_col(Col& Y, const Row& X, const ColQ<NB>& Ic,
                                                    int lo, int hi) {
    AccI<NB> t;
    mmi<NB, false>(t, X, Ic, lo, hi);
    to_colq(Y, t, lo, hi);
  }
};

// e = the smallest integer at which round-half-even(amax / 2^e) <= 127
// (frexp: amax = m 2^p with m in [0.5, 1) gives amax / 2^(p - 7) = 128 m,
// which rounds past 127 when 128 m >= 127.5), 0 for amax = 0
__device__ __forceinline__ int quant_exp(float amax) {
  int e = 0;
  if (amax > 0.f) {
    int p;
    const float mant = frexpf(amax, &p);
    e = p - 7 + (mant * 128.f >= 127.5f ? 1 : 0);
  }
  return e;
}

}  // namespace i8
}  // namespace gdn
