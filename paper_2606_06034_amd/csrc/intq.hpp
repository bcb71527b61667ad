// intq.hpp -- integer operands of the low-bit inverse paths on gfx950's
// int8 MFMA (v_mfma_i32_16x16x64_i8): int8 "quad" fragments of lower
// block-triangular C x C matrices (C = 16, 32, 64), their exact int32
// products, the identity, band masks and a wave-wide maximum.
//
// A quad holds 16 int8 per lane, four 16 x 16 blocks of 4 bytes: row quad
// R[I] = blocks (I, 0..3) in row form, column quad Cq[J] = blocks (0..3, J)
// in column form (the fragment forms of tile16.hpp); one MFMA contracts all
// four k-blocks (zero blocks where K > I or K < J).  C = 16, 32 use the
// leading one or two blocks.  Values are held as int32 blocks AccI between
// products (index bidx(I, J) of the lower blocks).
#pragma once

#include "tile16.hpp"

// wave reductions of the ROCm device library
extern "C" __device__ __attribute__((const)) int __ockl_wfred_max_i32(int);
extern "C" __device__ __attribute__((const)) float __ockl_wfred_max_f32(float);

namespace gdn {
namespace iq {

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
// The integer inverse of one tile (Section 3.5, Algorithm 1, in the integer
// arithmetic the library reads from Appendix G): from Lm = -A as codes (row
// form, strictly lower) with exponent eL, the masked Neumann powers
// B_n = M(B_{n-1} Lm) summed into N0 (band 1..N), E = Lm + Lm N0 - N0 (band
// 1..N set to its exact value 0), the residual powers P_s = E P_{s-1} summed
// into Gs, and T = N0 + Gs + N0 Gs; every product requantised, every sum
// exact in production order.  Returns the strict part of T_hat as codes Tr
// (row form) and its exponent eTo.  NC, SC >= 0 fix N and S at compile time
// (every band and block skip is then resolved by the compiler); -1 takes
// them from Nrt, Srt.
//
// Ops<NB> supplies one code width: fragment types Row, Col (operands in row
// and column form), Prod (an exact product) and Sum (an exact running sum);
// kQB and kAccB, log2 bounds of a code's and a product's magnitude; to_row,
// to_col (codes to fragments), mm<OUTQ> (exact product, blocks outside a
// band zero), band, requant (product to codes), requant_codes, row_to_col,
// col_to_row (form changes through the identity), rs_init, rs_add, rs_band,
// rs_finish.  Every helper visits only the blocks that can meet the band of
// sub-diagonals it is given; the other blocks are zero by the structure of
// the computation.
template <template <int> class Ops, int NB, int NC = -1, int SC = -1>
__device__ __forceinline__ void int_engine(const AccI<NB>& Lr, int eL, int Nrt, int Srt,
                                           AccI<NB>& Tr, int& eTo) {
  using O = Ops<NB>;
  constexpr int C = 16 * NB;
  constexpr int QB = O::kQB, ACCB = O::kAccB;
  const int N = NC >= 0 ? NC : Nrt;
  const int S = SC >= 0 ? SC : Srt;
  RowQ<NB> Iq;
  ColQ<NB> Ic;
  eye_quads(Iq, Ic);

  const bool nzL = amax_of(Lr, 1, C - 1) > 0;
  typename O::Row LRq;
  O::to_row(LRq, Lr, 1, C - 1);
  typename O::Col LCq;
  O::row_to_col(LCq, nullptr, LRq, Ic, 1, C - 1);

  // ---- N0 = sum of the masked powers B_n = M(B_{n-1} Lm) (band n..N), row form
  typename O::Sum ns;
  O::rs_init(ns, 1, N);
  if (N >= 1) {
    AccI<NB> B = Lr;
    band_i<NB, false>(B, 1, N);
    int eB;
    bool nzB;
    O::requant_codes(B, 1, N, eL, eB, nzB);
    O::rs_add(ns, B, 1, N, eB, QB, nzB);
    typename O::Row Bq;
    O::to_row(Bq, B, 1, N);
    auto power = [&](int n) {
      typename O::Prod D;
      O::template mm<true>(D, Bq, LCq, n, N);
      O::band(D, n, N);
      AccI<NB> q;
      O::requant(D, q, n, N, eB + eL, eB, nzB);
      O::rs_add(ns, q, n, N, eB, QB, nzB);
      O::to_row(Bq, q, n, N);
    };
    if constexpr (NC >= 0) {
#pragma unroll
      for (int n = 2; n <= NC; ++n) power(n);
    } else {
      for (int n = 2; n <= N; ++n) power(n);
    }
  }
  AccI<NB> N0r;
  int eN0;
  bool nzN0;
  O::rs_finish(ns, N0r, eN0, nzN0);
  typename O::Row N0q;
  O::to_row(N0q, N0r, 1, N);
  typename O::Col N0c;
  O::row_to_col(N0c, nullptr, N0q, Ic, 1, N);

  // ---- E = Lm + Lm N0 - N0 (row form), band 1..N zeroed
  typename O::Row ERq;
  typename O::Col ECq;
  AccI<NB> Ecol;
  int eE;
  bool nzE;
  {
    typename O::Prod LN;
    O::template mm<true>(LN, LRq, N0c, 2, C - 1);
    typename O::Sum es;
    O::rs_init(es, 1, C - 1);
    O::rs_add(es, Lr, 1, C - 1, eL, QB, nzL);
    O::rs_add(es, LN, 2, C - 1, eL + eN0, ACCB, nzL && nzN0);
    O::rs_add(es, N0r, 1, N, eN0, QB, nzN0, true);
    O::rs_band(es, N + 1, C - 1);
    AccI<NB> Er;
    O::rs_finish(es, Er, eE, nzE);
    O::to_row(ERq, Er, N + 1, C - 1);
    O::row_to_col(ECq, &Ecol, ERq, Ic, N + 1, C - 1);  // column form of E (exact codes)
  }

  // ---- residual powers P_s = E P_{s-1} (column form, band s(N+1)..), Gs = sum
  typename O::Sum gs;
  O::rs_init(gs, N + 1, C - 1);
  if (S >= 1) {
    O::rs_add(gs, Ecol, N + 1, C - 1, eE, QB, nzE);
    typename O::Col Pq = ECq;
    int eP = eE;
    bool nzP = nzE;
    auto chain = [&](int s) {
      const int lo = s * (N + 1);
      typename O::Prod D;
      O::template mm<false>(D, ERq, Pq, lo, C - 1);
      AccI<NB> q;
      O::requant(D, q, lo, C - 1, eE + eP, eP, nzP);
      O::rs_add(gs, q, lo, C - 1, eP, QB, nzP);
      O::to_col(Pq, q, lo, C - 1);
    };
    if constexpr (SC >= 0) {
#pragma unroll
      for (int s = 2; s <= SC; ++s) chain(s);
    } else {
      for (int s = 2; s <= S; ++s) chain(s);
    }
  }
  AccI<NB> Gc;
  int eG;
  bool nzG;
  O::rs_finish(gs, Gc, eG, nzG);
  typename O::Col GCq;
  O::to_col(GCq, Gc, N + 1, C - 1);
  AccI<NB> Gr;
  O::col_to_row(Gr, Iq, GCq, N + 1, C - 1);  // row form of Gs (exact codes)

  // ---- T = N0 + Gs + N0 Gs (row form), strict part
  bool nzT;
  {
    typename O::Prod NG;
    O::template mm<true>(NG, N0q, GCq, N + 2, C - 1);
    typename O::Sum ts;
    O::rs_init(ts, 1, C - 1);
    O::rs_add(ts, N0r, 1, N, eN0, QB, nzN0);
    O::rs_add(ts, Gr, N + 1, C - 1, eG, QB, nzG);
    O::rs_add(ts, NG, N + 2, C - 1, eN0 + eG, ACCB, nzN0 && nzG);
    O::rs_band(ts, 1, C - 1);
    O::rs_finish(ts, Tr, eTo, nzT);
  }
}

}  // namespace iq
}  // namespace gdn
