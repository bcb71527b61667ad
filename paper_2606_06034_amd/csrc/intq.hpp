// intq.hpp -- integer operands of the low-bit inverse paths on gfx950's
// int8 MFMA (v_mfma_i32_16x16x64_i8): int8 "quad" fragments of lower
// block-triangular C x C matrices (C = 16, 32, 64), their exact int32
// products, the identity, band masks, a wave-wide maximum, the scale rule
// of the quantiser, exact sums in fp64, and the integer inverse of one tile
// (int_engine) that both code widths run.
//
// A quad holds 16 int8 per lane, four 16 x 16 blocks of 4 bytes: row quad
// R[I] = blocks (I, 0..3) in row form, column quad Cq[J] = blocks (0..3, J)
// in column form (the fragment forms of tile16.hpp); one MFMA contracts all
// four k-blocks (zero blocks where K > I or K < J).  C = 16, 32 use the
// leading one or two blocks.  Values are held as int32 blocks AccI between
// products (index bidx(I, J) of the lower blocks).
#pragma once

#include "tile16.hpp"

#include <stdint.h>

// wave reductions of the ROCm device library
extern "C" __device__ __attribute__((const)) int __ockl_wfred_max_i32(int);
extern "C" __device__ __attribute__((const)) float __ockl_wfred_max_f32(float);

namespace gdn {
namespace iq {

typedef double f64x4 __attribute__((ext_vector_type(4)));

struct Quad {
  i32x4 v;  // dword K = 4 bytes of block K
};

template <int NB> struct RowQ { Quad r[NB]; };
template <int NB> struct ColQ { Quad c[NB]; };
template <int NB> struct AccI { i32x4 a[nlower(NB)]; };

__device__ __forceinline__ i32x4 zero_i4() { return i32x4{0, 0, 0, 0}; }

// 4 int32 in [-128, 127] <-> 4 bytes (value v in byte v)
__device__ __forceinline__ int pack4(i32x4 x) {
  return (int)((uint32_t)(x[0] & 0xff) | ((uint32_t)(x[1] & 0xff) << 8) |
               ((uint32_t)(x[2] & 0xff) << 16) | ((uint32_t)(x[3] & 0xff) << 24));
}
__device__ __forceinline__ i32x4 unpack4(int w) {
  i32x4 r;
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (int)(int8_t)(w >> (8 * v));
  return r;
}

template <int NB>
__device__ __forceinline__ i32x4 blki(const AccI<NB>& D, int I, int J) {
  return (J <= I && I < NB) ? D.a[bidx(I, J)] : zero_i4();
}
// Quads from blocks; blocks that cannot meet the band [lo, hi] (structurally
// zero) are packed as constant zeros.
template <int NB>
__device__ __forceinline__ void to_rowq(RowQ<NB>& X, const AccI<NB>& D, int lo = 0,
                                        int hi = 16 * NB) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int K = 0; K < 4; ++K)
      X.r[I].v[K] = (K <= I && I < NB && blk_nz(I - K, lo, hi)) ? pack4(D.a[bidx(I, K)]) : 0;
}
template <int NB>
__device__ __forceinline__ void to_colq(ColQ<NB>& Y, const AccI<NB>& D, int lo = 0,
                                        int hi = 16 * NB) {
#pragma unroll
  for (int J = 0; J < NB; ++J)
#pragma unroll
    for (int K = 0; K < 4; ++K)
      Y.c[J].v[K] = (K >= J && K < NB && blk_nz(K - J, lo, hi)) ? pack4(D.a[bidx(K, J)]) : 0;
}

// D = X Y (lower), blocks outside [olo, ohi] set to 0; OUTQ: row-form result.
template <int NB, bool OUTQ>
__device__ __forceinline__ void mmi(AccI<NB>& D, const RowQ<NB>& X, const ColQ<NB>& Y, int olo,
                                    int ohi) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      i32x4 acc = zero_i4();
      if (blk_nz(I - J, olo, ohi))
        acc = OUTQ ? __builtin_amdgcn_mfma_i32_16x16x64_i8(Y.c[J].v, X.r[I].v, acc, 0, 0, 0)
                   : __builtin_amdgcn_mfma_i32_16x16x64_i8(X.r[I].v, Y.c[J].v, acc, 0, 0, 0);
      D.a[bidx(I, J)] = acc;
    }
}

// identity as quads (row and column quads coincide)
template <int NB>
__device__ __forceinline__ void eye_quads(RowQ<NB>& R, ColQ<NB>& Cq) {
  AccI<NB> e;
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) e.a[b] = zero_i4();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int v = 0; v < 4; ++v) e.a[bidx(I, I)][v] = (c == 4 * g + v) ? 1 : 0;
  to_rowq(R, e);
  to_colq(Cq, e);
}

// zero entries outside lo <= i - j <= hi of the lower blocks a[bidx(I, J)]
// (any four-element block type)
template <int NB, bool COLFORM, typename V>
__device__ __forceinline__ void band_blocks(V* a, int lo, int hi) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      if (!blk_nz(I - J, lo, hi)) {
        a[bidx(I, J)] = V{};
      } else if (!blk_all_in(I - J, lo, hi)) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int d = COLFORM ? dcol(I - J, v) : drow(I - J, v);
          if (d < lo || d > hi) a[bidx(I, J)][v] = 0;
        }
      }
    }
}
template <int NB, bool COLFORM>
__device__ __forceinline__ void band_i(AccI<NB>& D, int lo, int hi) {
  band_blocks<NB, COLFORM>(D.a, lo, hi);
}

// wave-wide maximum (the device library's DPP reduction), as a scalar
__device__ __forceinline__ int wave_max(int x) {
  return __builtin_amdgcn_readfirstlane(__ockl_wfred_max_i32(x));
}

// max |D| over the blocks that can meet the band [lo, hi] (every other block
// is zero by the structure of the computation), wave-wide
template <int NB>
__device__ __forceinline__ int amax_of(const AccI<NB>& D, int lo, int hi) {
  int m = 0;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      if (blk_nz(I - J, lo, hi))
#pragma unroll
        for (int v = 0; v < 4; ++v) m = max(m, abs(D.a[bidx(I, J)][v]));
  return wave_max(m);
}


// ---------------------------------------------------------------------------
// Full 64 x 64 matrices (all 4 x 4 blocks; the off-diagonal block of a
// C = 128 tile), values as int32 blocks, block (I, J) at 4 I + J.

struct FullI {
  i32x4 a[16];
};

__device__ __forceinline__ void to_rowq_full(RowQ<4>& X, const FullI& D) {
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int K = 0; K < 4; ++K) X.r[I].v[K] = pack4(D.a[4 * I + K]);
}
// D in column form
__device__ __forceinline__ void to_colq_full(ColQ<4>& Y, const FullI& D) {
#pragma unroll
  for (int J = 0; J < 4; ++J)
#pragma unroll
    for (int K = 0; K < 4; ++K) Y.c[J].v[K] = pack4(D.a[4 * K + J]);
}
// D = X Y over the output block columns J0 .. J0 + JN - 1 (all 16 blocks
// by default; the other blocks of D are left as they are); X or Y may be
// lower: its quads carry the zero blocks.  OUTQ: row-form result.
template <bool OUTQ, int J0 = 0, int JN = 4>
__device__ __forceinline__ void mmi_full(FullI& D, const RowQ<4>& X, const ColQ<4>& Y) {
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = J0; J < J0 + JN; ++J)
      D.a[4 * I + J] =
          OUTQ ? __builtin_amdgcn_mfma_i32_16x16x64_i8(Y.c[J].v, X.r[I].v, zero_i4(), 0, 0, 0)
               : __builtin_amdgcn_mfma_i32_16x16x64_i8(X.r[I].v, Y.c[J].v, zero_i4(), 0, 0, 0);
}
__device__ __forceinline__ int amax_full(const FullI& D) {
  int m = 0;
#pragma unroll
  for (int b = 0; b < 16; ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) m = max(m, abs(D.a[b][v]));
  return wave_max(m);
}


// ---------------------------------------------------------------------------
// The scale rule.  A tensor of codes |q| <= Q with one power-of-two scale
// 2^e per tile; an exactly known tensor v is quantised to
// q = round-half-even(v / 2^e) with e the smallest integer at which no code
// leaves [-Q, Q], i.e. max|v| < (Q + 1/2) 2^e (Appendix G's
// q(x) = clip(round(x / Delta)) with the finest Delta = 2^e whose clip does
// nothing).  QB: 2^(QB - 1) <= Q < 2^QB.

// The shift s = e - e_v for values v = y 2^e_v held as integers y with
// max|y| = amax > 0 (int32): s is b - QB or b - QB + 1, b the bit length of
// amax (amax / 2^(b - QB) lies in [2^(QB-1), 2^QB)).
template <int Q, int QB>
__device__ __forceinline__ int shift_canon(int amax) {
  const int b = 32 - __clz(amax);
  const int s = b - QB;
  const bool over = s <= 0 ? ((int64_t)amax << -s) > Q
                           : 2 * (int64_t)amax >= ((2 * (int64_t)Q + 1) << s);
  return s + (over ? 1 : 0);
}

// The same shift from the high dword of max|y| for y held as fp64 integers
// (amax_hi > 0).  The test amax < (Q + 1/2) 2^s compares with a threshold
// of at most 16 significant bits, whose low dword is zero, so amax and its
// high dword (the value with the low dword cleared) compare alike with it.
// amax = m 2^p, m in [0.5, 1): 2^QB m < Q + 1/2 gives s = p - QB, else
// p - QB + 1.
template <int Q, int QB>
__device__ __forceinline__ int shift_canon_hi(int amax_hi) {
  const double a = __hiloint2double(amax_hi, 0);
  int p;
  const double m = frexp(a, &p);
  return p - QB + (m * (double)(1 << QB) >= (double)Q + 0.5 ? 1 : 0);
}

// round-half-even(x sc) as int32 for an fp64 integer x and a power of two sc
// with |x sc| < 2^31: x sc + 1.5 2^52 lies in [2^52, 2^53), where the fp64
// spacing is 1, so the fused addition rounds x sc half to even and the low
// dword of the sum holds the result in two's complement (1.5 2^52 has a zero
// low dword)
constexpr double kRoundMagic = 6755399441055744.0;  // 1.5 * 2^52
__device__ __forceinline__ int rne_scaled(double x, double sc) {
  return __double2loint(__builtin_fma(x, sc, kRoundMagic));
}

template <int NB> struct AccD { f64x4 a[nlower(NB)]; };  // fp64 integers

__device__ __forceinline__ double elem(const i32x4& x, int v) { return (double)x[v]; }
__device__ __forceinline__ double elem(const f64x4& x, int v) { return x[v]; }

// A term of an exact sum: the lower blocks of t (band [lo, hi]) times
// sign 2^e, absent when !p.  bits bounds |t| < 2^bits.
template <typename T> struct Term {
  const T* t;
  int e, bits, sign, lo, hi;
  bool p;
};

// the bit length of max|t| over the term's band (0 when t is zero): the
// wave maximum of the high dwords of |t| as fp64, whose frexp exponent is
// the bit length (an integer's high dword keeps its leading bit)
template <int NB, typename T>
__device__ __forceinline__ int term_bits(const Term<T>& x) {
  int mh = 0;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      if (blk_nz(I - J, x.lo, x.hi))
#pragma unroll
        for (int v = 0; v < 4; ++v) mh = max(mh, __double2hiint(fabs(elem(x.t->a[bidx(I, J)], v))));
  mh = wave_max(mh);
  if (mh == 0) return 0;
  int p;
  frexp(__hiloint2double(mh, 0), &p);
  return p;
}

// The exponent plan of an exact sum of up to three terms, wave-uniform:
// the scale of each present term relative to the finest one kept (emin),
// and which terms are rounded to the 52-bit window.  In: each term's
// exponent e, magnitude bits b (|t| < 2^b, 2^(b-1) <= max|t|) and presence
// p.  When the present terms span at most 52 bits the sum is exact in
// fp64.  Otherwise a term whose top lies QB + 6 bits or more under the
// coarsest top is dropped: unless the kept terms cancel below a quarter of
// the coarsest one's largest value, the output's quantum is at least
// 2^(top - QB - 2), so the dropped terms together stay below an eighth of
// it and move no code.  If the kept terms still span more than 52 bits, the
// finest are rounded to the window; exactness is claimed for neither of
// these two cases (no tile of the quantiser's output on the workloads
// reaches them).
struct SumPlan {
  int emin;
  bool p[3], r[3];
};
template <int QB>
__device__ __forceinline__ SumPlan sum_plan(const int (&e)[3], const int (&b)[3],
                                            const bool (&p)[3]) {
  SumPlan pl;
  int top = -(1 << 30), emin = 1 << 30;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    pl.p[k] = p[k];
    pl.r[k] = false;
    if (p[k]) {
      top = max(top, e[k] + b[k]);
      emin = min(emin, e[k]);
    }
  }
  if (top - emin > 52) {
    // only here are b the measured magnitudes (see exact_sum, sum2_full)
    emin = 1 << 30;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      pl.p[k] = p[k] && e[k] + b[k] > top - QB - 6;
      if (pl.p[k]) emin = min(emin, e[k]);
    }
  }
  if (top - emin > 52) {
    const int floor_e = top - 52;
    emin = 1 << 30;
#pragma unroll
    for (int k = 0; k < 3; ++k)
      if (pl.p[k]) {
        pl.r[k] = e[k] < floor_e;
        emin = min(emin, max(e[k], floor_e));
      }
  }
  pl.emin = emin;
  return pl;
}

// out = q(sum of the terms) over the blocks of the band [lo, hi]: the exact
// sum (every term aligned at the finest exponent among the kept ones)
// quantised once by the scale rule (Q, QB).  The values are fp64 integers.
// The plan first takes each term's bound bits; only when those span more
// than 52 bits are the terms' actual magnitudes measured (wave maxima), so
// that a zero or small term does not widen the window (sum_plan).  Returns
// the codes, their exponent and a non-zero flag; every block of out
// outside the band is set to 0.
template <int Q, int QB, int NB, typename T1, typename T2, typename T3>
__device__ __forceinline__ void exact_sum(AccI<NB>& out, int& eo, bool& nz, const Term<T1>& x,
                                          const Term<T2>& y, const Term<T3>& z, int lo, int hi) {
  int e[3] = {x.e, y.e, z.e}, b[3] = {x.bits, y.bits, z.bits};
  bool p[3] = {x.p, y.p, z.p};
  int emin = 1 << 30, top = -(1 << 30);
#pragma unroll
  for (int k = 0; k < 3; ++k)
    if (p[k]) {
      emin = min(emin, e[k]);
      top = max(top, e[k] + b[k]);
    }
  if (!p[0] && !p[1] && !p[2]) {
#pragma unroll
    for (int bb = 0; bb < nlower(NB); ++bb) out.a[bb] = zero_i4();
    eo = 0;
    nz = false;
    return;
  }
  if (top - emin > 52) {
    if (p[0]) { b[0] = term_bits<NB>(x); p[0] = b[0] > 0; }
    if (p[1]) { b[1] = term_bits<NB>(y); p[1] = b[1] > 0; }
    if (p[2]) { b[2] = term_bits<NB>(z); p[2] = b[2] > 0; }
  }
  const SumPlan pl = sum_plan<QB>(e, b, p);
  const double sx = pl.p[0] ? (double)x.sign * ldexp(1.0, x.e - pl.emin) : 0.0;
  const double sy = pl.p[1] ? (double)y.sign * ldexp(1.0, y.e - pl.emin) : 0.0;
  const double sz = pl.p[2] ? (double)z.sign * ldexp(1.0, z.e - pl.emin) : 0.0;
  auto val = [&](int I, int J, int v) {
    const int m = I - J, bi = bidx(I, J);
    double acc = 0.0;
    if (pl.p[0] && blk_nz(m, x.lo, x.hi)) {
      const double t = elem(x.t->a[bi], v) * sx;
      acc += pl.r[0] ? rint(t) : t;
    }
    if (pl.p[1] && blk_nz(m, y.lo, y.hi)) {
      const double t = elem(y.t->a[bi], v) * sy;
      acc += pl.r[1] ? rint(t) : t;
    }
    if (pl.p[2] && blk_nz(m, z.lo, z.hi)) {
      const double t = elem(z.t->a[bi], v) * sz;
      acc += pl.r[2] ? rint(t) : t;
    }
    return acc;
  };
  int mh = 0;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      if (blk_nz(I - J, lo, hi))
#pragma unroll
        for (int v = 0; v < 4; ++v) mh = max(mh, __double2hiint(fabs(val(I, J, v))));
  const int amax_hi = wave_max(mh);
  nz = amax_hi > 0;
  const int s = nz ? shift_canon_hi<Q, QB>(amax_hi) : 0;
  const double sc = ldexp(1.0, -s);
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      i32x4 r = zero_i4();
      if (nz && blk_nz(I - J, lo, hi))
#pragma unroll
        for (int v = 0; v < 4; ++v) r[v] = rne_scaled(val(I, J, v), sc);
      out.a[bidx(I, J)] = r;
    }
  eo = nz ? pl.emin + s : 0;
}

template <typename T>
__device__ __forceinline__ Term<T> term(const T& t, int e, int bits, int sign, int lo, int hi,
                                        bool p) {
  return Term<T>{&t, e, bits, sign, lo, hi, p};
}
template <typename T>
__device__ __forceinline__ Term<T> no_term(const T& t) {
  return Term<T>{&t, 0, 0, 1, 0, 0, false};
}

// Is every column sum of |E| (codes of a lower matrix in row form, band
// [lo, C-1], exponent e) at most 1?  Then |(P E)_ij| <= max|P| for any P,
// so each residual power is bounded by the one before it.  Lane (g, c) of
// a row-form block holds row c, columns 4g + v: the sum over a block's rows
// runs over the 16 lanes of one g (xor-shuffles 1, 2, 4, 8), the sum over
// block rows in the lane.
template <int NB>
__device__ __forceinline__ bool colsum_at_most_one(const AccI<NB>& E, int e, int lo) {
  int best = 0;
#pragma unroll
  for (int J = 0; J < NB; ++J)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      int sacc = 0;
#pragma unroll
      for (int I = J; I < NB; ++I)
        if (blk_nz(I - J, lo, 16 * NB - 1)) sacc += abs(E.a[bidx(I, J)][v]);
#pragma unroll
      for (int d = 1; d < 16; d <<= 1) sacc += __shfl_xor(sacc, d);
      best = max(best, sacc);
    }
  const int m = wave_max(best);
  if (m == 0) return true;
  if (e >= 0) return m <= 1 && e == 0;
  return -e >= 30 || m <= (1 << -e);
}

// identity codes (1 on the diagonal, exponent 0)
template <int NB>
__device__ __forceinline__ void eye_codes(AccI<NB>& D) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
#pragma unroll
      for (int v = 0; v < 4; ++v) D.a[bidx(I, J)][v] = (I == J && c == 4 * g + v) ? 1 : 0;
}

// ---------------------------------------------------------------------------
// The integer inverse of one tile: Algorithm 1 (Section 3.4) with integer
// activations (Section 3.5, Appendix G), every operator evaluated exactly
// from its operands' codes and its result quantised once by the scale rule:
//   P_1 = L (= -A), P_n = q(P_{n-1} L),          T0 = q(T0 + P_n),
//   T0 = M^(N) (.) T0 (codes masked, scale kept),
//   E = I - q((I + A) T0),
//   P_1 = E, P_s = q(P_{s-1} E),                 T = q(T + P_s),
//   T_hat = q(T0 T)
// (T0 starts at I, T at I).  Split form (PLAIN false): the unit diagonal of
// T0, T and T_hat stays out of the codes, so their tensors are the strict
// lower parts and a product of two of them is (I + X)(I + Y) = I + (X + Y +
// X Y), one rounding of the three-term sum; E = -q(A + N0 + A N0).  Plain
// form: every tensor holds its diagonal; E = q(I - q(T0 + A T0)).
//
// In: Lm = -A as codes (row form, strictly lower) with exponent eL.  Out:
// T_hat's tensor as codes Tr (row form) and its exponent eTo.  NC, SC >= 0
// fix N and S at compile time; -1 takes them from Nrt, Srt.
//
// Ops<NB> supplies one code width: fragment types Row, Col (operands in row
// and column form) and Prod (an exact product); kQ, kQB (the code range and
// its bits), kAccB (log2 bound of a product's magnitude); to_row, to_col
// (codes to fragments), codes (fragments back to codes), mm<OUTQ> (exact
// product, blocks outside a band zero), requant (a product to codes by the
// scale rule), canon (codes to the
// finest scale that holds them), add (q of the sum of two tensors of codes,
// the first known to be at its finest scale or not),
// row_to_col (column-form fragments of a row-form one, through the
// identity).  Every helper visits only the blocks that can meet the band of
// sub-diagonals it is given; the other blocks are zero by the structure of
// the computation.
template <template <int> class Ops, int NB, bool PLAIN, int NC = -1, int SC = -1>
__device__ __forceinline__ void int_engine(const AccI<NB>& Lr, int eL, int Nrt, int Srt,
                                           AccI<NB>& Tr, int& eTo) {
  using O = Ops<NB>;
  constexpr int C = 16 * NB;
  constexpr int Q = O::kQ, QB = O::kQB, ACCB = O::kAccB;
  constexpr int U0 = PLAIN ? 0 : 1;  // lowest sub-diagonal of T0's, T's and T_hat's tensors
  const int N = NC >= 0 ? NC : Nrt;
  const int S = SC >= 0 ? SC : Srt;
  RowQ<NB> Iq;
  ColQ<NB> Ic;
  eye_quads(Iq, Ic);

  const bool nzL = amax_of(Lr, 1, C - 1) > 0;
  typename O::Row LRq;
  O::to_row(LRq, Lr, 1, C - 1);
  typename O::Col LCq;
  O::row_to_col(LCq, LRq, Ic, 1, C - 1);

  // ---- T0 = sum_{n=0}^{N} L^n, then masked
  AccI<NB> T0;
  int eT0 = 0;
  bool nzT0 = PLAIN;
  if constexpr (PLAIN) eye_codes(T0);
  else {
#pragma unroll
    for (int b = 0; b < nlower(NB); ++b) T0.a[b] = zero_i4();
  }
  if (N >= 1) {
    AccI<NB> P = Lr;
    int eP = eL;
    bool nzP = nzL;
    O::canon(P, 1, C - 1, eP, nzP);
    O::add(T0, eT0, nzT0, U0, !PLAIN, P, eP, nzP, 1, 1, U0, C - 1);
    typename O::Row PRq;
    auto power = [&](int n) {
      O::to_row(PRq, P, n - 1, C - 1);
      typename O::Prod D;
      O::template mm<true>(D, PRq, LCq, n, C - 1);
      O::requant(D, P, n, C - 1, eP + eL, eP, nzP);
      O::add(T0, eT0, nzT0, U0, true, P, eP, nzP, 1, n, U0, C - 1);
    };
    if constexpr (NC >= 0) {
#pragma unroll
      for (int n = 2; n <= NC; ++n) power(n);
    } else {
      for (int n = 2; n <= N; ++n) power(n);
    }
  }
  band_i<NB, false>(T0, U0, N);
  nzT0 = amax_of(T0, U0, N) > 0;
  typename O::Row T0Rq;
  O::to_row(T0Rq, T0, U0, N);
  typename O::Col T0Cq;
  O::row_to_col(T0Cq, T0Rq, Ic, U0, N);

  // ---- E = I - q((I + A) T0), with (I + A) T0 = T0 - Lm T0
  constexpr int E0 = PLAIN ? 0 : 1;  // lowest sub-diagonal of E
  AccI<NB> E;
  int eE;
  bool nzE;
  {
    typename O::Prod D;
    O::template mm<true>(D, LRq, T0Cq, U0 + 1, C - 1);  // Lm T0
    if constexpr (!PLAIN) {
      // E = -(A + N0 + A N0) = Lm - N0 + Lm N0
      exact_sum<Q, QB, NB>(E, eE, nzE, term(Lr, eL, QB, 1, 1, C - 1, nzL),
                           term(T0, eT0, QB, -1, 1, N, nzT0),
                           term(D, eL + eT0, ACCB, 1, 2, C - 1, nzL && nzT0), 1, C - 1);
    } else {
      AccI<NB> M;
      int eM;
      bool nzM;
      exact_sum<Q, QB, NB>(M, eM, nzM, term(T0, eT0, QB, 1, 0, N, nzT0), no_term(T0),
                           term(D, eL + eT0, ACCB, -1, 1, C - 1, nzL && nzT0), 0, C - 1);
      eye_codes(E);
      eE = 0;
      nzE = true;
      O::add(E, eE, nzE, 0, false, M, eM, nzM, -1, 0, 0, C - 1);
    }
  }
  typename O::Row ERq;
  O::to_row(ERq, E, E0, C - 1);
  typename O::Col ECq;
  O::row_to_col(ECq, ERq, Ic, E0, C - 1);

  // ---- T = sum_{s=0}^{S} E^s
  AccI<NB> R;
  int eR = 0;
  bool nzR = PLAIN;
  if constexpr (PLAIN) eye_codes(R);
  else {
#pragma unroll
    for (int b = 0; b < nlower(NB); ++b) R.a[b] = zero_i4();
  }
  if (S >= 1) {
    O::add(R, eR, nzR, U0, !PLAIN, E, eE, nzE, 1, E0, U0, C - 1);
    AccI<NB> P;
    int eP = eE;
    bool nzP = nzE;
    typename O::Row PRq = ERq;
    // Once a residual power adds nothing to T (its exponent 2 QB + 3 or
    // more under T's, so the add leaves T's codes as they are) and every
    // column sum of |E| is at most 1, every later power is no larger, its
    // exponent no higher, and its add leaves T as it is too: the chain
    // stops there with the result it would have reached.
    const bool contracting = colsum_at_most_one(E, eE, E0);
    bool done = false;
    auto chain = [&](int s) {
      if (done) return;
      const int lo = PLAIN ? 0 : s;
      typename O::Prod D;
      O::template mm<true>(D, PRq, ECq, lo, C - 1);
      O::requant(D, P, lo, C - 1, eP + eE, eP, nzP);
      const bool idle = !nzP || (nzR && eR - eP >= 2 * QB + 3);
      O::add(R, eR, nzR, U0, true, P, eP, nzP, 1, lo, U0, C - 1);
      done = idle && contracting;
      if (!done) O::to_row(PRq, P, lo, C - 1);
    };
    // a rolled loop: unrolled, the early exit keeps every iteration's
    // operands live at once and costs a wave per SIMD
#pragma unroll 1
    for (int s = 2; s <= S; ++s) {
      chain(s);
      if (done) break;
    }
  }

  // ---- T_hat = q(T0 T)
  typename O::Col RCq;
  {
    typename O::Row RRq;
    O::to_row(RRq, R, U0, C - 1);
    O::row_to_col(RCq, RRq, Ic, U0, C - 1);
  }
  typename O::Prod D;
  O::template mm<true>(D, T0Rq, RCq, PLAIN ? 0 : 2, C - 1);
  // T0's codes again, from its row fragments (they hold every code exactly;
  // keeping the unpacked copy alive across the residual chain would cost a
  // wave per SIMD)
  O::codes(T0, T0Rq, U0, N);
  if constexpr (!PLAIN) {
    bool nzT;
    exact_sum<Q, QB, NB>(Tr, eTo, nzT, term(T0, eT0, QB, 1, 1, N, nzT0),
                         term(R, eR, QB, 1, 1, C - 1, nzR),
                         term(D, eT0 + eR, ACCB, 1, 2, C - 1, nzT0 && nzR), 1, C - 1);
  } else {
    bool nzT;
    O::requant(D, Tr, 0, C - 1, eT0 + eR, eTo, nzT);
  }
}

}  // namespace iq
}  // namespace gdn
