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

}  // namespace iq
}  // namespace gdn
