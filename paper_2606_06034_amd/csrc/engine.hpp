// engine.hpp -- the MatMul-only approximate inverse of one C x C tile in the
// registers of one wave (Sections 3.1-3.4 and Algorithm 1 of arXiv
// 2606.06034), plus tile load/store helpers.
//
// With Lm = -A (strictly lower):
//   T0 = M^(N) (Hadamard) sum_{n=0}^{N} Lm^n          (mask keeps i - j <= N)
//   E  = I - (I + A) T0 = Lm T0 - (T0 - I), which vanishes on i - j <= N
//   T  = T0 sum_{s=0}^{S} E^s = T0 + T0 Gs,  Gs = E + E^2 + ... + E^S
//
// Schedule (products are X * Y with X in row pairs, Y in column pairs):
//   * T0 by Horner, H <- I + Lm H, the identity entering through the MFMA
//     accumulator and the band mask applied after every step (entries of
//     Lm H on i - j <= N only read entries of H on the band, so masking
//     early equals masking the finished sum);
//   * E = band_{i-j > N}(Lm T0) in both forms: on the band E is exactly 0,
//     and off the band T0 vanishes so Lm T0 is E there;
//   * the residual sum, either (GH) by Horner, R <- I + E R from R = I + E,
//     then T = T0 R; or as the chain of powers P_s = E P_{s-1} in column
//     form (the same powers as Algorithm 1's P E chain), Gs += P_s, where
//     E^s vanishes exactly on i - j < s (N + 1) and those blocks are
//     skipped, then T = T0 + T0 Gs with T0 entering through the MFMA
//     accumulator.  Both evaluate T0 sum_{s=0}^{S} E^s; Horner keeps one
//     matrix live instead of a power and a running sum (fewer registers)
//     at the price of the chain's structural skipping.
// F = bf16x4 rounds every MFMA operand to bf16 (products accumulate in fp32,
// sums and masks run in fp32); F = f32x4 computes in fp32 throughout.
// SMALLN: the caller guarantees N <= 15, so T0's band lies in the diagonal
// and first sub-diagonal blocks and everything beyond is compile-time zero.
// NC, SC >= 0 fix N and S at compile time (every block skip and mask is then
// resolved by the compiler); -1 takes them from the runtime arguments.
#pragma once

#include "tile16.hpp"

namespace gdn {

// ---------------------------------------------------------------------------
// 4-element global IO

__device__ __forceinline__ f32x4 load4(const float* p) { return *(const f32x4*)p; }
__device__ __forceinline__ f32x4 load4(const __bf16* p) {
  return __builtin_convertvector(*(const bf16x4*)p, f32x4);
}
__device__ __forceinline__ void store4(float* p, f32x4 x) { *(f32x4*)p = x; }
__device__ __forceinline__ void store4(__bf16* p, f32x4 x) {
  *(bf16x4*)p = __builtin_convertvector(x, bf16x4);
}
__device__ __forceinline__ float load1(const float* p) { return *p; }
__device__ __forceinline__ float load1(const __bf16* p) { return (float)*p; }

// T0 = M^(N) (Hadamard) sum Lm^n keeps 0 <= i - j <= N: true for the
// 16 x 16 blocks at block distance m = I - J that meet that band (SMALLN:
// N <= 15, so m <= 1).
template <bool SMALLN>
__device__ __forceinline__ bool in_t0_band(int m, int N) {
  if constexpr (SMALLN) {
    if (m > 1) return false;
  }
  return blk_nz(m, 0, N);
}

// Lm = -A of a row-major tile (row stride ldr) as row-form f32 blocks
// (lane (g, c) reads 4 consecutive entries of row 16I + c), and the column
// form (lane (g, c): rows 16I + 4g + v of column 16J + c) of the blocks in
// T0's band only, the ones the engine reads.  The column blocks come from the
// row blocks through an identity MFMA (Lr I, exact: each output is one entry
// times 1 plus zeros) instead of 2-byte gathers from memory: 9 % less time
// for the standalone inverse at C = 64 on MI355X.  Entries on and above the
// diagonal are taken as 0.
// the lower-triangle blocks of a tile as read (row form), for callers that
// issue several tiles' loads before computing on the first
template <int NB, typename TIO>
__device__ __forceinline__ void load_lower_raw(const TIO* __restrict__ a, int ldr, Acc<NB>& R) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) R.a[bidx(I, J)] = load4(a + (I * 16 + c) * ldr + J * 16 + 4 * g);
}

template <int NB, typename F, bool SMALLN>
__device__ __forceinline__ void neg_strict_from(const Acc<NB>& R, int N, Acc<NB>& Lr,
                                                Acc<NB>& Lc) {
  const Pair<F> Ic = Pair<F>::make(eye4(), zero4());
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      Lr.a[bidx(I, J)] = band_block<false>(-R.a[bidx(I, J)], I - J, 1, 16 * NB);
      Lc.a[bidx(I, J)] =
          in_t0_band<SMALLN>(I - J, N)
              ? Pair<F>::template mma<false>(Pair<F>::make(Lr.a[bidx(I, J)], zero4()), Ic, zero4())
              : zero4();
    }
}

template <int NB, typename F, bool SMALLN, typename TIO>
__device__ __forceinline__ void load_neg_strict(const TIO* __restrict__ a, int ldr, int N,
                                                Acc<NB>& Lr, Acc<NB>& Lc) {
  Acc<NB> R;
  load_lower_raw<NB>(a, ldr, R);
  neg_strict_from<NB, F, SMALLN>(R, N, Lr, Lc);
}

// Lm = -A as row-form blocks only
template <int NB>
__device__ __forceinline__ void neg_strict_row_from(const Acc<NB>& R, Acc<NB>& Lr) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      Lr.a[bidx(I, J)] = band_block<false>(-R.a[bidx(I, J)], I - J, 1, 16 * NB);
}

template <int NB, typename TIO>
__device__ __forceinline__ void load_neg_strict_row(const TIO* __restrict__ a, int ldr,
                                                    Acc<NB>& Lr) {
  Acc<NB> R;
  load_lower_raw<NB>(a, ldr, R);
  neg_strict_row_from<NB>(R, Lr);
}

// Store a unit lower-triangular tile from its row-form blocks (diagonal
// written as exactly 1, the upper triangle as 0).  ldr = row stride.
template <int NB, typename TIO>
__device__ __forceinline__ void store_unit_row(TIO* __restrict__ t, int ldr, const Acc<NB>& Tr,
                                               Lane ln = lane_here()) {
  const int g = ln.g(), c = ln.c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J) {
      f32x4 x = zero4();
      if (J < I) x = Tr.a[bidx(I, J)];
      if (J == I) {
        x = Tr.a[bidx(I, J)];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int d = drow(0, v, ln);
          x[v] = d > 0 ? x[v] : (d == 0 ? 1.f : 0.f);
        }
      }
      store4(t + (I * 16 + c) * ldr + J * 16 + 4 * g, x);
    }
}

// ---------------------------------------------------------------------------

// The approximate inverse.  In: Lm as row pairs (LR), column pairs (LC) and
// f32 column blocks (Lc; only T0's band blocks are read).  Out: Tr, the
// row-form blocks of T (strict part exact, diagonal blocks carry T0's unit
// diagonal; callers write the diagonal as 1).
template <int NB, typename F, bool SMALLN, int NC = -1, int SC = -1, bool GH = true>
__device__ __forceinline__ void neumann_engine(const RowP<NB, F>& LR, const Acc<NB>& Lc, int Nrt,
                                               int Srt, Acc<NB>& Tr, Lane ln = lane_here()) {
  constexpr int C = 16 * NB;
  const int N = NC >= 0 ? NC : Nrt;
  const int S = SC >= 0 ? SC : Srt;

  // ---- T0 = I + (band of Lm + Lm^2 + ... + Lm^N), Horner, column form
  Acc<NB> H;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 x = in_t0_band<SMALLN>(I - J, N) ? band_block<true>(Lc.a[bidx(I, J)], I - J, 1, N, ln)
                                             : zero4();
      if (I == J) x += eye4(ln);
      H.a[bidx(I, J)] = x;
    }
  ColP<NB, F> T0c;
  to_colp(T0c, H);
  auto horner_step = [&]() {
    Acc<NB> D;
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) D.a[bidx(I, J)] = (I == J) ? eye4(ln) : zero4();
    mm<NB, false, true>(D, LR, 1, C - 1, T0c, 0, N, 1, N);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        if (in_t0_band<SMALLN>(I - J, N))
          D.a[bidx(I, J)] = band_block<true>(D.a[bidx(I, J)], I - J, 0, N, ln);
        else
          D.a[bidx(I, J)] = zero4();
    to_colp(T0c, D);
  };
  if constexpr (NC >= 0) {
#pragma unroll
    for (int n = 2; n <= NC; ++n) horner_step();
  } else {
    for (int n = 2; n <= N; ++n) horner_step();
  }
  RowP<NB, F> T0R;
  {
    Acc<NB> t;
    col_to_row(t, T0c, 0, N, ln);
    to_rowp(T0R, t);
  }

  // ---- E = band_{i-j > N}(Lm T0), both forms (Section 3.4)
  RowP<NB, F> ER;
  Acc<NB> Ec;  // column form
  {
    Acc<NB> D;
    mm<NB, true, false>(D, LR, 1, C - 1, T0c, 0, N, N + 1, C - 1);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        D.a[bidx(I, J)] = band_block<false>(D.a[bidx(I, J)], I - J, N + 1, C - 1, ln);
    to_rowp(ER, D);
    mm<NB, false, false>(D, LR, 1, C - 1, T0c, 0, N, N + 1, C - 1);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        Ec.a[bidx(I, J)] = S >= 1 ? band_block<true>(D.a[bidx(I, J)], I - J, N + 1, C - 1, ln)
                                  : zero4();
  }

  if constexpr (GH) {
    // ---- R = I + E + ... + E^S by Horner, R <- I + E R (column pairs; the
    // identity enters through the MFMA accumulator).  E R only reaches
    // i - j >= N + 1, and R's upper triangle and band 1..N stay exact zeros,
    // so no mask is needed.  Holds R alone instead of a power and a sum.
    ColP<NB, F> RC;
#pragma unroll
    for (int I = 0; I < NB; ++I) Ec.a[bidx(I, I)] += eye4(ln);
    to_colp(RC, Ec);
    auto horner_r = [&]() {
      Acc<NB> D;
#pragma unroll
      for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int J = 0; J <= I; ++J) D.a[bidx(I, J)] = (I == J) ? eye4(ln) : zero4();
      mm<NB, false, true>(D, ER, N + 1, C - 1, RC, 0, C - 1, N + 1, C - 1);
      to_colp(RC, D);
    };
    if constexpr (SC >= 0) {
#pragma unroll
      for (int s = 2; s <= SC; ++s) horner_r();
    } else {
      for (int s = 2; s <= S; ++s) horner_r();
    }
    // ---- T = T0 R, row form
    mm<NB, true, false>(Tr, T0R, 0, N, RC, 0, C - 1, 0, C - 1);
  } else {
    // ---- residual powers P_s = E P_{s-1}, Gs = E + ... + E^S (column form)
    ColP<NB, F> P;
    Acc<NB> G = Ec;
    to_colp(P, G);
    auto chain_step = [&](int s) {
      const int plo = (s - 1) * (N + 1), lo = s * (N + 1);
      Acc<NB> D;
      mm<NB, false, false>(D, ER, N + 1, C - 1, P, plo, C - 1, lo, C - 1);
#pragma unroll
      for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int J = 0; J <= I; ++J)
          if (blk_nz(I - J, lo, C - 1)) {
            G.a[bidx(I, J)] += D.a[bidx(I, J)];
            pin(G.a[bidx(I, J)]);
          }
      to_colp(P, D);
    };
    if constexpr (SC >= 0) {
#pragma unroll
      for (int s = 2; s <= SC; ++s) chain_step(s);
    } else {
      for (int s = 2; s <= S; ++s) chain_step(s);
    }
    // ---- T = T0 + T0 Gs, row form; T0 (as rounded for the products)
    // enters through the accumulator
    ColP<NB, F> GC;
    to_colp(GC, G);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) {
        const int p = J >> 1;
        Tr.a[bidx(I, J)] = (J & 1) ? T0R.r[I][p].hi() : T0R.r[I][p].lo();
      }
    mm<NB, true, true>(Tr, T0R, 0, N, GC, N + 1, C - 1, N + 1, C - 1);
  }
}

// ---------------------------------------------------------------------------
// Exact inverse by blocks: the two-block recursion of Appendix E,
//   [[X_11, 0], [X_21, X_22]] with X_21 = X_22 L_21 X_11   (L = Lm = -A),
// taken all the way down.  Inside each 16 x 16 diagonal block it runs on
// masked 16 x 16 products: with O_k the entries of L that join two blocks
// of size 2^k into one of size 2^(k+1), and X_k the inverse of the part of
// (I - L) made of 2^k x 2^k diagonal blocks,
//   X_{k+1} = X_k + X_k O_k X_k        (X_1 = I + O_0),
// exact because O_k X_k O_k = 0; every intermediate is a principal
// sub-block of X, so nothing grows beyond the inverse itself.  Across the
// 16 x 16 blocks it continues as block forward substitution,
//   X_IJ = X_II sum_{K=J}^{I-1} L_IK X_KJ   (I > J, rows in order).
// Out: Tr, the row-form blocks of X (unit diagonal, zero upper triangle).

// entry (i, j) of a 16 x 16 block belongs to O_k
__device__ __forceinline__ bool in_level(int i, int j, int k) {
  return i > j && (i >> k) != (j >> k) && (i >> (k + 1)) == (j >> (k + 1));
}

template <int NB, typename F>
__device__ __forceinline__ void blockwise_inverse(const Acc<NB>& Lr, Acc<NB>& Tr,
                                                  Lane ln = lane_here()) {
  const int g = ln.g(), c = ln.c();
  const f32x4 e = eye4(ln);
  auto mk = [](f32x4 x) { return Pair<F>::make(x, zero4()); };
  const Pair<F> Ic = mk(e);
  f32x4 Xc[nlower(NB)];  // column form (right operands of later rows)
#pragma unroll
  for (int I = 0; I < NB; ++I) {
    const f32x4 lr = Lr.a[bidx(I, I)];
    const f32x4 lc = Pair<F>::template mma<false>(mk(lr), Ic, zero4());  // the block, column form
    // X_1 = I + O_0 in both forms (row form: i = c, j = 4g + v; column: i = 4g + v, j = c)
    f32x4 xr = e, xc = e;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if (in_level(c, 4 * g + v, 0)) xr[v] += lr[v];
      if (in_level(4 * g + v, c, 0)) xc[v] += lc[v];
    }
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      f32x4 oc;
#pragma unroll
      for (int v = 0; v < 4; ++v) oc[v] = in_level(4 * g + v, c, k) ? lc[v] : 0.f;
      const Pair<F> T = mk(Pair<F>::template mma<true>(mk(xr), mk(oc), zero4()));  // X_k O_k, row
      const Pair<F> Xk = mk(xc);
      const f32x4 nc = Pair<F>::template mma<false>(T, Xk, xc);
      const f32x4 nr = Pair<F>::template mma<true>(T, Xk, xr);
      xc = nc;
      xr = nr;
    }
    Tr.a[bidx(I, I)] = xr;
    Xc[bidx(I, I)] = xc;
  }
#pragma unroll
  for (int I = 1; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < I; ++J) {
      // S = sum_{K=J}^{I-1} L_IK X_KJ (column form), k-blocks paired
      f32x4 sc = zero4();
#pragma unroll
      for (int p = 0; p < npair(NB); ++p) {
        const int k0 = 2 * p, k1 = 2 * p + 1;
        const bool u0 = k0 >= J && k0 < I, u1 = k1 >= J && k1 < I;
        if (!u0 && !u1) continue;
        const Pair<F> x = Pair<F>::make(u0 ? Lr.a[bidx(I, k0)] : zero4(),
                                        u1 ? Lr.a[bidx(I, k1)] : zero4());
        const Pair<F> y = Pair<F>::make(u0 ? Xc[bidx(k0, J)] : zero4(),
                                        u1 ? Xc[bidx(k1, J)] : zero4());
        sc = Pair<F>::template mma<false>(x, y, sc);
      }
      const Pair<F> D = mk(Tr.a[bidx(I, I)]), Sc = mk(sc);
      Xc[bidx(I, J)] = Pair<F>::template mma<false>(D, Sc, zero4());
      Tr.a[bidx(I, J)] = Pair<F>::template mma<true>(D, Sc, zero4());
    }
}

}  // namespace gdn
