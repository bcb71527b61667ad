// int16_ops.hpp -- the INT16 arithmetic of the integer inverse (Section 3.5,
// Appendix G of arXiv 2606.06034): 16-bit codes as two int8 limbs, exact
// products in fp64, quantisation by the scale rule of intq.hpp, exact fp64
// sums and the I16Ops width the shared engine (int_engine of intq.hpp) runs
// on, plus the per-tile quantiser's exponent.  Used by int16.hip and by the
// layer forward's integer-inverse mode.
#pragma once

#include "intq.hpp"

namespace gdn {
namespace i16 {

using namespace iq;

constexpr int kQmax = 32639;

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

// a product (fp64 integers, exact) of exponent e_in to codes q by the scale
// rule over the band blocks (other blocks 0); exponent and non-zero flag
// through refs.  The wave maximum is taken over the high dwords of |x|
// (shift_canon_hi).
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
  nz = amax_hi > 0;
  const int s = nz ? shift_canon_hi<kQmax, 15>(amax_hi) : 0;
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
  e_out = nz ? e_in + s : 0;
}

// exact int32 values (|y| < 2^30) of exponent e_in to codes by the scale
// rule, in place: a right shift by s > 0 rounded half to even (the sum
// y + 2^(s-1) stays below 2^31), or an exact left shift; exponent and
// non-zero flag through refs
template <int NB>
__device__ __forceinline__ void requant_i32(AccI<NB>& D, int lo, int hi, int e_in, int& e_out,
                                            bool& nz) {
  const int amax = amax_of(D, lo, hi);
  nz = amax > 0;
  if (!nz) {
    e_out = 0;
    return;
  }
  const int s = shift_canon<kQmax, 15>(amax);
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      if (blk_nz(I - J, lo, hi))
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int y = D.a[bidx(I, J)][v];
          D.a[bidx(I, J)][v] =
              s > 0 ? (y + (1 << (s - 1)) - 1 + ((y >> s) & 1)) >> s : y << (-s);
        }
  e_out = e_in + s;
}

// codes (|q| <= 32639) to the finest scale that holds them (exact left
// shift), in place
template <int NB>
__device__ __forceinline__ void canon(AccI<NB>& q, int lo, int hi, int& e, bool& nz) {
  const int amax = amax_of(q, lo, hi);
  nz = amax > 0;
  if (!nz) {
    e = 0;
    return;
  }
  const int s = shift_canon<kQmax, 15>(amax);
  if (s < 0) {
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (blk_nz(I - J, lo, hi))
#pragma unroll
          for (int v = 0; v < 4; ++v) q.a[bidx(I, J)][v] <<= -s;
  }
  e += s;
}

// ---------------------------------------------------------------------------

// The INT16 width for the shared integer engine (int_engine of intq.hpp):
// limb quads, products as fp64 integers, sums exact in fp64.
template <int NB> struct I16Ops {
  using Row = RowL<NB>;
  using Col = ColL<NB>;
  using Prod = AccD<NB>;
  static constexpr int kQ = kQmax;
  static constexpr int kQB = 15;                                      // |code| < 2^15
  static constexpr int kAccB = 30 + (NB == 1 ? 4 : NB == 2 ? 5 : 6);  // |product| < C 2^30
  static __device__ __forceinline__ void to_row(Row& X, const AccI<NB>& D, int lo, int hi) {
    to_rowl(X, D, lo, hi);
  }
  static __device__ __forceinline__ void to_col(Col& Y, const AccI<NB>& D, int lo, int hi) {
    to_coll(Y, D, lo, hi);
  }
  // the codes 256 h + l of the blocks of X that can meet [lo, hi] (others 0)
  static __device__ __forceinline__ void codes(AccI<NB>& D, const Row& X, int lo, int hi) {
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        D.a[bidx(I, J)] = blk_nz(I - J, lo, hi)
                              ? unpack4(X.h.r[I].v[J]) * 256 + unpack4(X.l.r[I].v[J])
                              : zero_i4();
  }
  template <bool OUTQ>
  static __device__ __forceinline__ void mm(Prod& D, const Row& X, const Col& Y, int lo, int hi) {
    mml<NB, OUTQ>(D, X, Y, lo, hi);
  }
  static __device__ __forceinline__ void requant(const Prod& D, AccI<NB>& q, int lo, int hi,
                                                 int e_in, int& e_out, bool& nz) {
    i16::requant(D, q, lo, hi, e_in, e_out, nz);
  }
  static __device__ __forceinline__ void canon(AccI<NB>& q, int lo, int hi, int& e, bool& nz) {
    i16::canon(q, lo, hi, e, nz);
  }
  // X = q(X 2^eX + ys Y 2^eY) over [lo, hi] (X's band [xlo, hi], Y's
  // [ylo, hi]); Y is at the finest scale that holds it, and so is X when
  // xc.  Exponents 2 QB + 3 or more apart: the finer term is below an
  // eighth of the output quantum and leaves the coarser's codes as they are
  // (at their finest scale); at most QB apart: the aligned sum is below
  // 32639 (2^15 + 1) < 2^30 and exact in int32, and so is its rounding;
  // otherwise the sum is exact in fp64 (below 2^48).  Every path gives the
  // exact sum quantised once by the scale rule.
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
    if (g >= -kQB && g <= kQB) {
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
      requant_i32(X, lo, hi, e0, eX, nzX);
      return;
    }
    AccI<NB> out;
    exact_sum<kQ, kQB, NB>(out, eX, nzX, term(X, eX, kQB, 1, xlo, hi, nzX),
                           term(Y, eY, kQB, ys, ylo, hi, nzY), no_term(Y), lo, hi);
    X = out;
  }
  static __device__ __forceinline__ void row_to_col(Col& Y, const Row& X, const ColQ<NB>& Ic,
                                                    int lo, int hi) {
    i16::row_to_col<NB>(Y, nullptr, X, Ic, lo, hi);
  }
};

// e = the smallest integer at which round-half-even(amax / 2^e) <= 32639
// (frexp: amax = m 2^p with m in [0.5, 1) gives amax / 2^(p - 15) =
// 32768 m, which rounds past 32639 when 32768 m >= 32639.5), 0 for
// amax = 0
__device__ __forceinline__ int quant_exp(float amax) {
  int e = 0;
  if (amax > 0.f) {
    int p;
    const float mant = frexpf(amax, &p);
    e = p - 15 + (mant * 32768.f >= 32639.5f ? 1 : 0);
  }
  return e;
}

}  // namespace i16
}  // namespace gdn
