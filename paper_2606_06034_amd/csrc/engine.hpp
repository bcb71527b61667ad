// engine.hpp -- the MatMul-only approximate inverse of one C x C tile, held
// in the registers of one wave (Sections 3.1-3.4 and Algorithm 1 of
// arXiv 2606.06034), plus the tile load/store helpers.
//
// With Lm = -A (strictly lower):
//   T0 = I + N0,  N0 = M^(N) (Hadamard) sum_{n=1}^{N} Lm^n   (mask keeps i-j <= N)
//   E  = I - (I + A) T0 = Lm T0 - N0, which vanishes on i - j <= N
//   T  = T0 sum_{s=0}^{S} E^s = T0 + T0 (E + E^2 + ... + E^S)
//
// Schedule on the tile forms of tile16.hpp:
//   * powers P_n = Lm P_{n-1} in column form, only on the band blocks;
//   * T0 kept in column form (right factor of Lm T0) and in row form (left
//     factor of the final product; one identity-MFMA layout change);
//   * E computed in both forms directly from Lm (row) and T0 (column);
//     its band i - j <= N is set to its exact value 0, so E^s vanishes
//     exactly on i - j < s (N + 1) and those blocks are skipped;
//   * the residual powers run as P_s = E P_{s-1} (column form), the same
//     powers as Algorithm 1's P E chain;
//   * the final product T0 G is split as T0 + T0 Gs (Gs = G - I) so only the
//     small strict part is rounded when the operands are bf16.
// Operands F are bf16x4 (bf16 mode: every MFMA operand rounded to bf16) or
// f32x4 (fp32 mode).  Products, sums and the identity parts stay in fp32.
#pragma once

#include "tile16.hpp"

namespace gdn {

// ---------------------------------------------------------------------------
// 4-element global IO

__device__ __forceinline__ f32x4 load4(const float* p) { return *(const f32x4*)p; }
__device__ __forceinline__ f32x4 load4(const __bf16* p) { return to_f32(*(const bf16x4*)p); }
__device__ __forceinline__ void store4(float* p, f32x4 x) { *(f32x4*)p = x; }
__device__ __forceinline__ void store4(__bf16* p, f32x4 x) { *(bf16x4*)p = to_bf16(x); }

// Lm = -A in row form from a row-major tile with row stride ldr; entries on
// and above the diagonal are read as 0.
template <int NB, typename F, typename TIO>
__device__ __forceinline__ void load_neg_strict_row(const TIO* __restrict__ a, int ldr,
                                                    F (&LQ)[nlower(NB)]) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 x = load4(a + (I * 16 + c) * ldr + J * 16 + 4 * g);
#pragma unroll
      for (int v = 0; v < 4; ++v) x[v] = (dQ(I, J, v) > 0) ? -x[v] : 0.f;
      LQ[bidx(I, J)] = Op<F>::from(x);
    }
}

// Store a unit lower-triangular tile given its strict part in row form:
// diagonal written as exactly 1, upper triangle as 0.  ldr = row stride.
template <int NB, typename TIO>
__device__ __forceinline__ void store_unit_row(TIO* __restrict__ t, int ldr,
                                               const f32x4 (&Tr)[nlower(NB)]) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J) {
      f32x4 x = zero4();
      if (J <= I) {
        x = Tr[bidx(I, J)];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int d = dQ(I, J, v);
          x[v] = d > 0 ? x[v] : (d == 0 ? 1.f : 0.f);
        }
      }
      store4(t + (I * 16 + c) * ldr + J * 16 + 4 * g, x);
    }
}

// ---------------------------------------------------------------------------
// The approximate inverse.  In: Lm in row form (LQ) and column form (LC).
// Out: strict lower part of T in row form (Tr); T's unit diagonal is
// implicit (the caller writes it).

template <int NB, typename F>
__device__ __forceinline__ void neumann_engine(const F (&LQ)[nlower(NB)],
                                               const F (&LC)[nlower(NB)], int N, int S,
                                               f32x4 (&Tr)[nlower(NB)]) {
  constexpr int C = 16 * NB;
  constexpr int NL = nlower(NB);

  // ---- T0 = I + N0: masked truncated Neumann sum (Sections 3.1, 3.3)
  f32x4 N0c[NL];
  F Pc[NL];
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 x = Op<F>::f32(LC[bidx(I, J)]);
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (dP(I, J, v) > N) x[v] = 0.f;
      N0c[bidx(I, J)] = x;
      Pc[bidx(I, J)] = Op<F>::from(x);
    }
  for (int n = 2; n <= N; ++n) {
    f32x4 D[NL];
    lower_mm<NB, false>(D, LQ, 1, C - 1, Pc, n - 1, N, n, N);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) {
        f32x4 x = D[bidx(I, J)];
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (dP(I, J, v) > N) x[v] = 0.f;
        N0c[bidx(I, J)] += x;
        Pc[bidx(I, J)] = Op<F>::from(x);
      }
  }

  F T0c[NL], T0r[NL];
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 x = N0c[bidx(I, J)];
      if (I == J) x += eye4();
      T0c[bidx(I, J)] = Op<F>::from(x);
    }
  {
    f32x4 tmp[NL];
    to_row<NB>(tmp, T0c, 0, N);
    cvt_all<NB>(T0r, tmp);
  }

  // ---- E = Lm T0 - N0, exactly 0 on i - j <= N (Section 3.4)
  F Er[NL];
  f32x4 Gc[NL];  // strict part of G = sum_{s=0}^{S} E^s, column form
  {
    f32x4 D[NL];
    lower_mm<NB, false>(D, LQ, 1, C - 1, T0c, 0, N, N + 1, C - 1);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) {
        f32x4 x = D[bidx(I, J)];
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (dP(I, J, v) <= N || S < 1) x[v] = 0.f;
        Gc[bidx(I, J)] = x;
        Pc[bidx(I, J)] = Op<F>::from(x);
      }
    lower_mm<NB, true>(D, LQ, 1, C - 1, T0c, 0, N, N + 1, C - 1);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) {
        f32x4 x = D[bidx(I, J)];
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (dQ(I, J, v) <= N) x[v] = 0.f;
        Er[bidx(I, J)] = Op<F>::from(x);
      }
  }

  // ---- residual powers P_s = E P_{s-1}, accumulated into Gs
  for (int s = 2; s <= S; ++s) {
    f32x4 D[NL];
    lower_mm<NB, false>(D, Er, N + 1, C - 1, Pc, (s - 1) * (N + 1), C - 1, s * (N + 1), C - 1);
#pragma unroll
    for (int b = 0; b < NL; ++b) {
      Gc[b] += D[b];
      Pc[b] = Op<F>::from(D[b]);
    }
  }

  // ---- T = T0 + T0 Gs, row form
  F Gf[NL];
  cvt_all<NB>(Gf, Gc);
  lower_mm<NB, true>(Tr, T0r, 0, N, Gf, N + 1, C - 1, N + 1, C - 1);
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 t0 = Op<F>::f32(T0r[bidx(I, J)]);
      if (I == J) t0 -= eye4();
      Tr[bidx(I, J)] += t0;
    }
}

}  // namespace gdn
