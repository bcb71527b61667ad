// int16_ops.hpp -- the INT16 arithmetic of the integer inverse (Section 3.5,
// Appendix G of arXiv 2606.06034): 16-bit codes as two int8 limbs, exact
// products in fp64, requantisation, exact fp64 running sums and the I16Ops
// width the shared engine (int_engine of intq.hpp) runs on, plus the
// per-tile quantiser's exponent.  Used by int16.hip and by the layer
// forward's integer-inverse mode.
#pragma once

#include "intq.hpp"

namespace gdn {
namespace i16 {

using namespace iq;

constexpr int kQmax = 32639;
constexpr int kAlignBits = 31;

typedef double f64x4 __attribute__((ext_vector_type(4)));

template <int NB> struct AccD { f64x4 a[nlower(NB)]; };  // fp64 integers

// the two int8 limbs of a matrix of codes, as quads
template <int NB> struct RowL { RowQ<NB> h, l; };
template <int NB> struct ColL { ColQ<NB> h, l; };

// The limb bytes of a code c = 256 h + l (l in [-128, 127]): l's byte is
// byte 0 of c, and c + 128 = 256 h + (l + 128) with 0 <= l + 128 <= 255, so
// h's byte is byte 1 of c + 128.  Four codes of a block give one dword of a
// quad per limb.
__device__ __forceinline__ int pack_lo(i32x4 c) {
  return (int)(((uint32_t)c[0] & 0xffu) | (((uint32_t)c[1] & 0xffu) << 8) |
               (((uint32_t)c[2] & 0xffu) << 16) | ((uint32_t)c[3] << 24));
}
__device__ __forceinline__ int pack_hi(i32x4 c) {
  const i32x4 u = c + 128;
  return (int)((((uint32_t)u[0] >> 8) & 0xffu) | ((uint32_t)u[1] & 0xff00u) |
               (((uint32_t)u[2] & 0xff00u) << 8) | (((uint32_t)u[3] & 0xff00u) << 16));
}

// limb quads of the blocks that can meet [lo, hi] (others zero), row form
template <int NB>
__device__ __forceinline__ void to_rowl(RowL<NB>& X, const AccI<NB>& D, int lo, int hi) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int K = 0; K < 4; ++K) {
      const bool live = K <= I && I < NB && blk_nz(I - K, lo, hi);
      X.h.r[I].v[K] = live ? pack_hi(D.a[bidx(I, K)]) : 0;
      X.l.r[I].v[K] = live ? pack_lo(D.a[bidx(I, K)]) : 0;
    }
}
// the same in column form
template <int NB>
__device__ __forceinline__ void to_coll(ColL<NB>& Y, const AccI<NB>& D, int lo, int hi) {
#pragma unroll
  for (int J = 0; J < NB; ++J)
#pragma unroll
    for (int K = 0; K < 4; ++K) {
      const bool live = K >= J && K < NB && blk_nz(K - J, lo, hi);
      Y.h.c[J].v[K] = live ? pack_hi(D.a[bidx(K, J)]) : 0;
      Y.l.c[J].v[K] = live ? pack_lo(D.a[bidx(K, J)]) : 0;
    }
}

// D = X Y exactly, blocks outside [olo, ohi] set to 0; OUTQ: row-form result
template <int NB, bool OUTQ>
__device__ __forceinline__ void mml(AccD<NB>& D, const RowL<NB>& X, const ColL<NB>& Y, int olo,
                                    int ohi) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f64x4 r = f64x4{0.0, 0.0, 0.0, 0.0};
      if (blk_nz(I - J, olo, ohi)) {
        const i32x4 xh = X.h.r[I].v, xl = X.l.r[I].v, yh = Y.h.c[J].v, yl = Y.l.c[J].v;
        const i32x4 z = zero_i4();
        i32x4 hh, mx, ll;
        if constexpr (OUTQ) {
          hh = __builtin_amdgcn_mfma_i32_16x16x64_i8(yh, xh, z, 0, 0, 0);
          mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(yl, xh, z, 0, 0, 0);
          mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(yh, xl, mx, 0, 0, 0);
          ll = __builtin_amdgcn_mfma_i32_16x16x64_i8(yl, xl, z, 0, 0, 0);
        } else {
          hh = __builtin_amdgcn_mfma_i32_16x16x64_i8(xh, yh, z, 0, 0, 0);
          mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(xh, yl, z, 0, 0, 0);
          mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(xl, yh, mx, 0, 0, 0);
          ll = __builtin_amdgcn_mfma_i32_16x16x64_i8(xl, yl, z, 0, 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v)
          r[v] = __builtin_fma((double)(hh[v] * 256 + mx[v]), 256.0, (double)ll[v]);
      }
      D.a[bidx(I, J)] = r;
    }
}

// codes of the limb matrices recombined: D = 256 H + L
template <int NB>
__device__ __forceinline__ void join(AccI<NB>& D, const AccI<NB>& H, const AccI<NB>& L) {
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) D.a[b] = H.a[b] * 256 + L.a[b];
}

// Form changes through the identity, limb by limb (exact).
// Column-form limbs (and, when wanted, codes) of a row-form matrix.
template <int NB>
__device__ __forceinline__ void row_to_col(ColL<NB>& Y, AccI<NB>* codes, const RowL<NB>& X,
                                           const ColQ<NB>& Ic, int lo, int hi) {
  AccI<NB> h, l;
  mmi<NB, false>(h, X.h, Ic, lo, hi);
  mmi<NB, false>(l, X.l, Ic, lo, hi);
  to_colq(Y.h, h, lo, hi);
  to_colq(Y.l, l, lo, hi);
  if (codes) join(*codes, h, l);
}
// Row-form codes of a column-form matrix.
template <int NB>
__device__ __forceinline__ void col_to_row(AccI<NB>& D, const RowQ<NB>& Iq, const ColL<NB>& Y,
                                           int lo, int hi) {
  AccI<NB> h, l;
  mmi<NB, true>(h, Iq, Y.h, lo, hi);
  mmi<NB, true>(l, Iq, Y.l, lo, hi);
  join(D, h, l);
}

// Smallest s >= 0 with round-half-even(amax / 2^s) <= 32639, from the high
// dword of amax (an fp64 integer >= 0, lo dword dropped).  The test is
// amax < 32639.5 2^s; the threshold has 16 significant bits, so its low
// dword is zero and amax and its truncation to the high dword compare
// alike with it.  amax = m 2^p, m in [0.5, 1): 2^15 m < 32639.5 gives
// s = p - 15, else p - 14 (never below 0).
__device__ __forceinline__ int shift_for_hi(int amax_hi) {
  const double a = __hiloint2double(amax_hi, 0);
  int p;
  const double m = frexp(a, &p);
  return max(0, p - 15 + (m * 32768.0 >= 32639.5 ? 1 : 0));
}

// round-half-even(x) as int32 for an fp64 x with |x| < 2^31: x + 1.5 2^52
// lies in [2^52, 2^53), where the fp64 spacing is 1, so the addition (fused
// with the scaling) rounds x half to even and the low dword of the sum holds
// the result in two's complement (1.5 2^52 has a zero low dword)
constexpr double kRoundMagic = 6755399441055744.0;  // 1.5 * 2^52
__device__ __forceinline__ int rne_scaled(double x, double sc) {
  return __double2loint(__builtin_fma(x, sc, kRoundMagic));
}

// requantise the band blocks of the fp64 integers D to codes q (other blocks
// 0); exponent and non-zero flag through refs
template <int NB>
__device__ __forceinline__ void requant(const AccD<NB>& D, AccI<NB>& q, int lo, int hi, int e_in,
                                        int& e_out, bool& nz) {
  int m = 0;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      if (blk_nz(I - J, lo, hi))
#pragma unroll
        for (int v = 0; v < 4; ++v) m = max(m, __double2hiint(fabs(D.a[bidx(I, J)][v])));
  const int amax_hi = wave_max(m);
  const int s = shift_for_hi(amax_hi);
  const double sc = ldexp(1.0, -s);
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      i32x4 r = zero_i4();
      if (blk_nz(I - J, lo, hi))
#pragma unroll
        for (int v = 0; v < 4; ++v) r[v] = rne_scaled(D.a[bidx(I, J)][v], sc);
      q.a[bidx(I, J)] = r;
    }
  nz = amax_hi > 0;
  e_out = nz ? e_in + s : 0;
}
// the same for a matrix of codes (|q| <= 32639: never shifted)
template <int NB>
__device__ __forceinline__ void requant_codes(const AccI<NB>& q, int lo, int hi, int e_in,
                                              int& e_out, bool& nz) {
  nz = amax_of(q, lo, hi) > 0;
  e_out = nz ? e_in : 0;
}

// exact running fp64 sum over the band [lo, hi] (the union of its terms')
template <int NB> struct RunSum {
  AccD<NB> acc;
  int e;
  bool any;
  int lo, hi;
};
template <int NB>
__device__ __forceinline__ void rs_init(RunSum<NB>& R, int lo, int hi) {
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) R.acc.a[b] = f64x4{0.0, 0.0, 0.0, 0.0};
  R.e = 0;
  R.any = false;
  R.lo = lo;
  R.hi = hi;
}
template <int NB>
__device__ __forceinline__ f64x4 as_f64(const AccI<NB>& t, int b) {
  return __builtin_convertvector(t.a[b], f64x4);
}
template <int NB>
__device__ __forceinline__ f64x4 as_f64(const AccD<NB>& t, int b) {
  return t.a[b];
}
// add the term t (codes or fp64 integers; band [tlo, thi] inside the sum's)
// of exponent et, |t| < 2^bits
template <int NB, typename Term>
__device__ __forceinline__ void rs_add(RunSum<NB>& R, const Term& t, int tlo, int thi, int et,
                                       int bits, bool present, bool negate = false) {
  if (!present) return;
  const int top = et + bits - kAlignBits;
  if (!R.any) {
    R.e = top;
    R.any = true;
  } else if (top > R.e) {
    const double sc = ldexp(1.0, R.e - top);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (blk_nz(I - J, R.lo, R.hi))
#pragma unroll
          for (int v = 0; v < 4; ++v)
            R.acc.a[bidx(I, J)][v] = rint(R.acc.a[bidx(I, J)][v] * sc);
    R.e = top;
  }
  // a wave-uniform shift: exact scaling when it is >= 0, else rounded in
  const int sh = et - R.e;
  const double sc = negate ? -ldexp(1.0, sh) : ldexp(1.0, sh);
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      if (blk_nz(I - J, tlo, thi)) {
        const f64x4 x = as_f64<NB>(t, bidx(I, J));
        if (sh >= 0) {
#pragma unroll
          for (int v = 0; v < 4; ++v)
            R.acc.a[bidx(I, J)][v] = __builtin_fma(x[v], sc, R.acc.a[bidx(I, J)][v]);
        } else {
#pragma unroll
          for (int v = 0; v < 4; ++v) R.acc.a[bidx(I, J)][v] += rint(x[v] * sc);
        }
      }
}

template <int NB>
__device__ __forceinline__ void rs_finish(const RunSum<NB>& R, AccI<NB>& q, int& e, bool& nz) {
  requant(R.acc, q, R.lo, R.hi, R.any ? R.e : 0, e, nz);
}

// ---------------------------------------------------------------------------

// The INT16 width for the shared integer engine (int_engine of intq.hpp):
// limb quads, products and running sums as fp64 integers.
template <int NB> struct I16Ops {
  using Row = RowL<NB>;
  using Col = ColL<NB>;
  using Prod = AccD<NB>;
  using Sum = RunSum<NB>;
  static constexpr int kQB = 15;                                      // |code| < 2^15
  static constexpr int kAccB = 30 + (NB == 1 ? 4 : NB == 2 ? 5 : 6);  // |product| < C 2^30
  static __device__ __forceinline__ void to_row(Row& X, const AccI<NB>& D, int lo, int hi) {
    to_rowl(X, D, lo, hi);
  }
  static __device__ __forceinline__ void to_col(Col& Y, const AccI<NB>& D, int lo, int hi) {
    to_coll(Y, D, lo, hi);
  }
  template <bool OUTQ>
  static __device__ __forceinline__ void mm(Prod& D, const Row& X, const Col& Y, int lo, int hi) {
    mml<NB, OUTQ>(D, X, Y, lo, hi);
  }
  static __device__ __forceinline__ void band(Prod& D, int lo, int hi) {
    band_blocks<NB, false>(D.a, lo, hi);
  }
  static __device__ __forceinline__ void requant(const Prod& D, AccI<NB>& q, int lo, int hi,
                                                 int e_in, int& e_out, bool& nz) {
    i16::requant(D, q, lo, hi, e_in, e_out, nz);
  }
  static __device__ __forceinline__ void requant_codes(const AccI<NB>& q, int lo, int hi,
                                                       int e_in, int& e_out, bool& nz) {
    i16::requant_codes(q, lo, hi, e_in, e_out, nz);
  }
  static __device__ __forceinline__ void row_to_col(Col& Y, AccI<NB>* codes, const Row& X,
                                                    const ColQ<NB>& Ic, int lo, int hi) {
    i16::row_to_col<NB>(Y, codes, X, Ic, lo, hi);
  }
  static __device__ __forceinline__ void col_to_row(AccI<NB>& D, const RowQ<NB>& Iq,
                                                    const Col& Y, int lo, int hi) {
    i16::col_to_row<NB>(D, Iq, Y, lo, hi);
  }
  static __device__ __forceinline__ void rs_init(Sum& R, int lo, int hi) {
    i16::rs_init(R, lo, hi);
  }
  template <typename Term>
  static __device__ __forceinline__ void rs_add(Sum& R, const Term& t, int tlo, int thi, int et,
                                                int bits, bool present, bool negate = false) {
    i16::rs_add(R, t, tlo, thi, et, bits, present, negate);
  }
  static __device__ __forceinline__ void rs_band(Sum& R, int lo, int hi) {
    band_blocks<NB, false>(R.acc.a, lo, hi);
    R.lo = lo;
  }
  static __device__ __forceinline__ void rs_finish(const Sum& R, AccI<NB>& q, int& e, bool& nz) {
    i16::rs_finish(R, q, e, nz);
  }
};

// e = the smallest integer with amax / 2^e <= 32639 (frexp: amax = m 2^p
// with m in [0.5, 1) gives amax / 2^(p - 15) = 32768 m), 0 for amax = 0
__device__ __forceinline__ int quant_exp(float amax) {
  int e = 0;
  if (amax > 0.f) {
    int p;
    const float mant = frexpf(amax, &p);
    e = p - 15 + (mant * 32768.f > 32639.f ? 1 : 0);
  }
  return e;
}

}  // namespace i16
}  // namespace gdn
