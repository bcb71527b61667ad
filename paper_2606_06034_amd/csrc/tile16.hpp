// tile16.hpp -- register-resident lower-triangular C x C tiles on gfx950 MFMA.
//
// A C x C matrix is cut into 16 x 16 blocks (NB = C / 16 per side).  A block
// lives in one of two fragment forms of the 16 x 16 MFMA family (lane l,
// g = l >> 4, c = l & 15, four values v = 0..3 per lane):
//
//   column form: lane (g, c) holds M[4g + v][c]  -- the accumulator layout of
//                v_mfma_*_16x16*, and the B-operand layout;
//   row form:    lane (g, c) holds M[c][4g + v]  -- the A-operand layout.
//
// An MFMA computes D = X * Y from X in row form and Y in column form and
// leaves D in column form; swapping the operands computes D^T = Y^T X^T from
// the same fragments, which leaves D in row form.  Both factors index their
// k-slots identically (k = 4g + v of a 16-wide block), so chained products
// never leave registers.
//
// Operands are kept as PAIR fragments over the fixed k-pairs {2p, 2p + 1}:
//   row form    X[I][p] = [X(I, 2p), X(I, 2p + 1)]   (zero where K > I)
//   column form Y[p][J] = [Y(2p, J), Y(2p + 1, J)]   (zero where K < J)
// so one v_mfma_f32_16x16x32_bf16 contracts a whole pair with no operand
// shuffling; a pair holding a single live block carries a zero half.  Every
// bf16 product uses this one opcode: chaining a 16x16x16 bf16 MFMA onto a
// 16x16x32 accumulator (SrcC = the previous result) got no wait states from
// this toolchain and read a stale accumulator on gfx950.
//
// Structural zeros: a matrix whose entries vanish outside the sub-diagonals
// lo <= i - j <= hi skips every block that cannot meet that band (a block
// at block-subdiagonal m spans i - j in [16m - 15, 16m + 15]).  Entries that
// vanish inside a computed block are exact zeros by construction, so the
// skipping is exact (NaN/Inf inputs aside).
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
__host__ __device__ constexpr int npair(int NB) { return (NB + 1) / 2; }

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int lane_g() { return (threadIdx.x & 63) >> 4; }
__device__ __forceinline__ int lane_c() { return threadIdx.x & 15; }

// The lane coordinates the lane-dependent helpers work from, passed as a
// defaulted last argument so a caller can hand one set down a call chain.
struct Lane {
  int id;
  __device__ __forceinline__ int g() const { return id >> 4; }
  __device__ __forceinline__ int c() const { return id & 15; }
};
__device__ __forceinline__ Lane lane_here() { return Lane{(int)(threadIdx.x & 63)}; }

// Can a block at block-subdiagonal m hold entries with lo <= i - j <= hi?
__device__ __forceinline__ bool blk_nz(int m, int lo, int hi) {
  return (16 * m + 15 >= lo) && (16 * m - 15 <= hi);
}
// Is every entry of such a block inside [lo, hi]?
__device__ __forceinline__ bool blk_all_in(int m, int lo, int hi) {
  return (16 * m - 15 >= lo) && (16 * m + 15 <= hi);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Materialise a value at this point of the program.  Used on running sums
// so the compiler cannot sink their additions to the last use and keep
// every addend alive until then.
__device__ __forceinline__ void pin(f32x4& x) { asm volatile("" : "+v"(x)); }

// identity block (both forms coincide)
__device__ __forceinline__ f32x4 eye4(Lane ln = lane_here()) {
  const int g = ln.g(), c = ln.c();
  f32x4 r;
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (c == 4 * g + v) ? 1.f : 0.f;
  return r;
}

// i - j of value v of this lane in a block at block-subdiagonal m
__device__ __forceinline__ int dcol(int m, int v, Lane ln = lane_here()) {
  return 16 * m + 4 * ln.g() + v - ln.c();
}
__device__ __forceinline__ int drow(int m, int v, Lane ln = lane_here()) {
  return 16 * m + ln.c() - 4 * ln.g() - v;
}

// Zero the entries of a block outside [lo, hi]; scalar tests skip the VALU
// work for blocks entirely inside (kept) or outside (zeroed) the band.
template <bool COLFORM>
__device__ __forceinline__ f32x4 band_block(f32x4 x, int m, int lo, int hi,
                                            Lane ln = lane_here()) {
  if (!blk_nz(m, lo, hi)) return zero4();
  if (blk_all_in(m, lo, hi)) return x;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int d = COLFORM ? dcol(m, v, ln) : drow(m, v, ln);
    x[v] = (d >= lo && d <= hi) ? x[v] : 0.f;
  }
  return x;
}

// ---------------------------------------------------------------------------
// pair fragments

template <typename F> struct Pair;

template <> struct Pair<bf16x4> {  // bf16 compute
  bf16x8 v;
  static __device__ __forceinline__ Pair make(f32x4 lo, f32x4 hi) {
    const bf16x4 a = __builtin_convertvector(lo, bf16x4);
    const bf16x4 b = __builtin_convertvector(hi, bf16x4);
    return Pair{__builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7)};
  }
  static __device__ __forceinline__ Pair zero() { return make(zero4(), zero4()); }
  __device__ __forceinline__ f32x4 lo() const {
    return __builtin_convertvector(__builtin_shufflevector(v, v, 0, 1, 2, 3), f32x4);
  }
  __device__ __forceinline__ f32x4 hi() const {
    return __builtin_convertvector(__builtin_shufflevector(v, v, 4, 5, 6, 7), f32x4);
  }
  // D += X Y (OUTQ: result in row form)
  template <bool OUTQ>
  static __device__ __forceinline__ f32x4 mma(const Pair& x, const Pair& y, f32x4 acc) {
    if constexpr (OUTQ)
      return __builtin_amdgcn_mfma_f32_16x16x32_bf16(y.v, x.v, acc, 0, 0, 0);
    else
      return __builtin_amdgcn_mfma_f32_16x16x32_bf16(x.v, y.v, acc, 0, 0, 0);
  }
};

template <> struct Pair<f32x4> {  // fp32 compute: eight 16x16x4 MFMAs per pair
  f32x4 a, b;
  static __device__ __forceinline__ Pair make(f32x4 lo, f32x4 hi) { return Pair{lo, hi}; }
  static __device__ __forceinline__ Pair zero() { return Pair{zero4(), zero4()}; }
  __device__ __forceinline__ f32x4 lo() const { return a; }
  __device__ __forceinline__ f32x4 hi() const { return b; }
  template <bool OUTQ>
  static __device__ __forceinline__ f32x4 mma(const Pair& x, const Pair& y, f32x4 acc) {
#pragma unroll
    for (int v = 0; v < 4; ++v)
      acc = OUTQ ? __builtin_amdgcn_mfma_f32_16x16x4f32(y.a[v], x.a[v], acc, 0, 0, 0)
                 : __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[v], y.a[v], acc, 0, 0, 0);
#pragma unroll
    for (int v = 0; v < 4; ++v)
      acc = OUTQ ? __builtin_amdgcn_mfma_f32_16x16x4f32(y.b[v], x.b[v], acc, 0, 0, 0)
                 : __builtin_amdgcn_mfma_f32_16x16x4f32(x.b[v], y.b[v], acc, 0, 0, 0);
    return acc;
  }
};

// Lower block-triangular matrices as pair fragments.
template <int NB, typename F> struct RowP {
  Pair<F> r[NB][npair(NB)];
};
template <int NB, typename F> struct ColP {
  Pair<F> c[npair(NB)][NB];
};
template <int NB> struct Acc {  // f32 lower blocks, index bidx(I, J)
  f32x4 a[nlower(NB)];
};

template <int NB>
__device__ __forceinline__ f32x4 blk(const Acc<NB>& D, int I, int J) {
  return (J <= I && I < NB) ? D.a[bidx(I, J)] : zero4();
}

// Row-form pairs from row-form f32 blocks (zero above the diagonal).
template <int NB, typename F>
__device__ __forceinline__ void to_rowp(RowP<NB, F>& X, const Acc<NB>& D) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int p = 0; p < npair(NB); ++p)
      X.r[I][p] = (2 * p <= I) ? Pair<F>::make(blk(D, I, 2 * p), blk(D, I, 2 * p + 1))
                               : Pair<F>::zero();
}
// Column-form pairs from column-form f32 blocks.
template <int NB, typename F>
__device__ __forceinline__ void to_colp(ColP<NB, F>& Y, const Acc<NB>& D) {
#pragma unroll
  for (int p = 0; p < npair(NB); ++p)
#pragma unroll
    for (int J = 0; J < NB; ++J)
      Y.c[p][J] = (2 * p + 1 >= J) ? Pair<F>::make(blk(D, 2 * p, J), blk(D, 2 * p + 1, J))
                                   : Pair<F>::zero();
}

// ---------------------------------------------------------------------------
// D (+)= X * Y for lower block-triangular X (row pairs, entries on sub-
// diagonals [xlo, xhi]) and Y (column pairs, [ylo, yhi]); only blocks that
// can meet [olo, ohi] are computed, the others are set to 0 (or left alone
// when ACCUM).  OUTQ selects the result form.  All bounds are wave-uniform.

template <int NB, bool OUTQ, bool ACCUM, typename F>
__device__ __forceinline__ void mm(Acc<NB>& D, const RowP<NB, F>& X, int xlo, int xhi,
                                   const ColP<NB, F>& Y, int ylo, int yhi, int olo, int ohi) {
  const int dlo = max(xlo + ylo, olo), dhi = min(xhi + yhi, ohi);
#pragma unroll
  for (int I = 0; I < NB; ++I) {
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 acc = ACCUM ? D.a[bidx(I, J)] : zero4();
      if (blk_nz(I - J, dlo, dhi)) {
#pragma unroll
        for (int p = 0; p < npair(NB); ++p) {
          const int k0 = 2 * p, k1 = 2 * p + 1;
          if (k0 > I || k1 < J) continue;
          const bool a0 = k0 >= J && blk_nz(I - k0, xlo, xhi) && blk_nz(k0 - J, ylo, yhi);
          const bool a1 = k1 <= I && k1 < NB && blk_nz(I - k1, xlo, xhi) &&
                          blk_nz(k1 - J, ylo, yhi);
          if (a0 || a1) acc = Pair<F>::template mma<OUTQ>(X.r[I][p], Y.c[p][J], acc);
        }
      }
      D.a[bidx(I, J)] = acc;
    }
  }
}

// Layout changes through the identity: row form of a column-form matrix
// (Z = I Z, row result) and column form of a row-form matrix (Z = Z I).
template <int NB, typename F>
__device__ __forceinline__ void col_to_row(Acc<NB>& D, const ColP<NB, F>& Z, int lo, int hi,
                                           Lane ln = lane_here()) {
  RowP<NB, F> id;
  Acc<NB> e;
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) e.a[b] = zero4();
#pragma unroll
  for (int I = 0; I < NB; ++I) e.a[bidx(I, I)] = eye4(ln);
  to_rowp(id, e);
  mm<NB, true, false>(D, id, 0, 0, Z, lo, hi, lo, hi);
}
template <int NB, typename F>
__device__ __forceinline__ void row_to_col(Acc<NB>& D, const RowP<NB, F>& Z, int lo, int hi,
                                           Lane ln = lane_here()) {
  ColP<NB, F> id;
  Acc<NB> e;
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) e.a[b] = zero4();
#pragma unroll
  for (int I = 0; I < NB; ++I) e.a[bidx(I, I)] = eye4(ln);
  to_colp(id, e);
  mm<NB, false, false>(D, Z, lo, hi, id, 0, 0, lo, hi);
}

}  // namespace gdn
