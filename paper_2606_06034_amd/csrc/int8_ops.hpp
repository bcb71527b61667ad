// int8_ops.hpp -- the INT8 arithmetic of the integer inverse (Section 3.5,
// Appendix G of arXiv 2606.06034): round-half-even shifts, requantisation,
// exact int32 running sums and the I8Ops width the shared engine
// (int_engine of intq.hpp) runs on, plus the per-tile quantiser's exponent.
// Used by int8.hip and by the layer forward's integer-inverse mode.
#pragma once

#include "intq.hpp"

namespace gdn {
namespace i8 {

using namespace iq;

constexpr int kAlignBits = 23;

// round-half-even(y / 2^s) for 1 <= s <= 30 and |y| < 2^30 (every value
// here stays below 2^24)
__device__ __forceinline__ int rne_pos(int y, int s) {
  return (y + (1 << (s - 1)) - 1 + ((y >> s) & 1)) >> s;
}
// any s >= 0 (s >= 31 rounds every |y| < 2^30 to 0)
__device__ __forceinline__ int rne_sh(int y, int s) {
  if (s <= 0) return y;
  if (s >= 31) return 0;
  return rne_pos(y, s);
}

// every entry rounded by a wave-uniform shift s >= 1
template <int NB>
__device__ __forceinline__ void shift_all(AccI<NB>& D, int s) {
  if (s >= 31) {
#pragma unroll
    for (int b = 0; b < nlower(NB); ++b) D.a[b] = zero_i4();
    return;
  }
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) D.a[b][v] = rne_pos(D.a[b][v], s);
}

// The helpers below visit only the blocks that can meet a band [lo, hi] of
// sub-diagonals; every other block of their operand is exactly zero by the
// structure of the computation, so skipping it changes no result.

// smallest s >= 0 with rne(amax / 2^s) <= 127
__device__ __forceinline__ int shift_for(int amax) {
  if (amax <= 127) return 0;
  int s = (32 - __clz(amax)) - 7;
  if (rne_sh(amax, s) > 127) ++s;
  return s;
}

// every entry rounded by a wave-uniform shift s >= 1
template <int NB>
__device__ __forceinline__ void shift_all(AccI<NB>& D, int s, int lo, int hi) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      if (blk_nz(I - J, lo, hi)) {
        if (s >= 31) {
          D.a[bidx(I, J)] = zero_i4();
        } else {
#pragma unroll
          for (int v = 0; v < 4; ++v) D.a[bidx(I, J)][v] = rne_pos(D.a[bidx(I, J)][v], s);
        }
      }
}

// requantise in place; returns (new exponent, non-zero flag) through refs
template <int NB>
__device__ __forceinline__ void requant(AccI<NB>& D, int lo, int hi, int e_in, int& e_out,
                                        bool& nz) {
  const int amax = amax_of(D, lo, hi);
  const int s = shift_for(amax);
  if (s > 0) shift_all(D, s, lo, hi);
  nz = amax > 0;
  e_out = nz ? e_in + s : 0;
}

// exact running int32 sum over the band [lo, hi] (the union of its terms')
template <int NB> struct RunSum {
  AccI<NB> acc;
  int e;
  bool any;
  int lo, hi;
};
template <int NB>
__device__ __forceinline__ void rs_init(RunSum<NB>& R, int lo, int hi) {
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) R.acc.a[b] = zero_i4();
  R.e = 0;
  R.any = false;
  R.lo = lo;
  R.hi = hi;
}
// add the term t (band [tlo, thi] inside the sum's) of exponent et, |t| < 2^bits
template <int NB>
__device__ __forceinline__ void rs_add(RunSum<NB>& R, const AccI<NB>& t, int tlo, int thi,
                                       int et, int bits, bool present, bool negate = false) {
  if (!present) return;
  const int top = et + bits - kAlignBits;
  if (!R.any) {
    R.e = top;
    R.any = true;
  } else if (top > R.e) {
    shift_all(R.acc, top - R.e, R.lo, R.hi);
    R.e = top;
  }
  // the shift is wave-uniform: one branch, not a select per entry
  const int sh = et - R.e;
  if (sh >= 0) {
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (blk_nz(I - J, tlo, thi))
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int x = negate ? -t.a[bidx(I, J)][v] : t.a[bidx(I, J)][v];
            R.acc.a[bidx(I, J)][v] += x << sh;
          }
  } else if (sh > -31) {
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (blk_nz(I - J, tlo, thi))
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int x = negate ? -t.a[bidx(I, J)][v] : t.a[bidx(I, J)][v];
            R.acc.a[bidx(I, J)][v] += rne_pos(x, -sh);
          }
  }
}

template <int NB>
__device__ __forceinline__ void rs_finish(RunSum<NB>& R, AccI<NB>& q, int& e, bool& nz) {
  q = R.acc;
  requant(q, R.lo, R.hi, R.any ? R.e : 0, e, nz);
}

// ---------------------------------------------------------------------------

// The INT8 width for the shared integer engine (int_engine of intq.hpp):
// quads, exact int32 products, int32 running sums.
template <int NB> struct I8Ops {
  using Row = RowQ<NB>;
  using Col = ColQ<NB>;
  using Prod = AccI<NB>;
  using Sum = RunSum<NB>;
  static constexpr int kQB = 7;                                       // |code| < 2^7
  static constexpr int kAccB = 14 + (NB == 1 ? 4 : NB == 2 ? 5 : 6);  // |product| < C 2^14
  static __device__ __forceinline__ void to_row(Row& X, const AccI<NB>& D, int lo, int hi) {
    to_rowq(X, D, lo, hi);
  }
  static __device__ __forceinline__ void to_col(Col& Y, const AccI<NB>& D, int lo, int hi) {
    to_colq(Y, D, lo, hi);
  }
  template <bool OUTQ>
  static __device__ __forceinline__ void mm(Prod& D, const Row& X, const Col& Y, int lo, int hi) {
    mmi<NB, OUTQ>(D, X, Y, lo, hi);
  }
  static __device__ __forceinline__ void band(Prod& D, int lo, int hi) {
    band_i<NB, false>(D, lo, hi);
  }
  // the product is requantised in place and handed on as the codes
  static __device__ __forceinline__ void requant(Prod& D, AccI<NB>& q, int lo, int hi, int e_in,
                                                 int& e_out, bool& nz) {
    i8::requant(D, lo, hi, e_in, e_out, nz);
    q = D;
  }
  static __device__ __forceinline__ void requant_codes(AccI<NB>& q, int lo, int hi, int e_in,
                                                       int& e_out, bool& nz) {
    i8::requant(q, lo, hi, e_in, e_out, nz);
  }
  static __device__ __forceinline__ void row_to_col(Col& Y, AccI<NB>* codes, const Row& X,
                                                    const ColQ<NB>& Ic, int lo, int hi) {
    AccI<NB> t;
    mmi<NB, false>(t, X, Ic, lo, hi);
    to_colq(Y, t, lo, hi);
    if (codes) *codes = t;
  }
  static __device__ __forceinline__ void col_to_row(AccI<NB>& D, const RowQ<NB>& Iq,
                                                    const Col& Y, int lo, int hi) {
    mmi<NB, true>(D, Iq, Y, lo, hi);
  }
  static __device__ __forceinline__ void rs_init(Sum& R, int lo, int hi) { i8::rs_init(R, lo, hi); }
  static __device__ __forceinline__ void rs_add(Sum& R, const AccI<NB>& t, int tlo, int thi,
                                                int et, int bits, bool present,
                                                bool negate = false) {
    i8::rs_add(R, t, tlo, thi, et, bits, present, negate);
  }
  static __device__ __forceinline__ void rs_band(Sum& R, int lo, int hi) {
    band_i<NB, false>(R.acc, lo, hi);
    R.lo = lo;
  }
  static __device__ __forceinline__ void rs_finish(Sum& R, AccI<NB>& q, int& e, bool& nz) {
    i8::rs_finish(R, q, e, nz);
  }
};

// e = the smallest integer with amax / 2^e <= 127 (frexp: amax = m 2^p with
// m in [0.5, 1) gives amax / 2^(p - 7) = 128 m), 0 for amax = 0
__device__ __forceinline__ int quant_exp(float amax) {
  int e = 0;
  if (amax > 0.f) {
    int p;
    const float mant = frexpf(amax, &p);
    e = p - 7 + (mant * 128.f > 127.f ? 1 : 0);
  }
  return e;
}

}  // namespace i8
}  // namespace gdn
