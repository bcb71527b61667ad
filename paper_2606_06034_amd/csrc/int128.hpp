// int128.hpp -- the integer inverse at C = 128, block-wise (Appendix E of
// arXiv 2606.06034, with the 64 x 64 blocks that Appendix H names as the
// smallest for the integer settings), for either code width.
//
// A C = 128 tile of codes holds three blocks with an exponent each, in the
// order (11, 21, 22): the strict lower parts of the two diagonal blocks and
// the whole block 21 (block 12 of a lower-triangular tile is zero).
//
// Inverse, two waves per tile: wave w inverts diagonal block w with the
// one-tile engine (int_engine, X_ww = I + N_ww), then the off-diagonal block
// is formed from the right by two MatMuls,
//   P = A21 X11 = A21 + A21 N11,      X21 = -(X22 P) = -(P + N22 P),
// each the exact sum of its code term and its exact product, quantised once
// by the scale rule (intq.hpp); each wave forms two of the four 16-column
// block columns of P and X21, the diagonal blocks and the maxima of the
// quantisations passing through LDS.
//
// W (one code width) supplies: Code (the storage type), load4 / store4 (four
// consecutive codes <-> i32x4), qexp (the quantiser's exponent of a block
// maximum), engine<NC, SC> (the one-tile inverse of a 64 x 64 block), Row,
// Col, to_row, to_col (the engine's fragments of lower matrices), to_frow
// (row-form fragments of a full matrix), frow_to_col (row-form fragments to
// column-form ones, exact), FProd and fmm<OUTQ, J0, JN> (an exact product
// over the output block columns J0 .. J0 + JN - 1) and codes (the codes of
// one block of row-form fragments), besides the engine width's kQ, kQB and
// kAccB.
#pragma once

#include "chunk.hpp"
#include "intq.hpp"

namespace gdn {
namespace iq {

// Tdeq of a diagonal block (row stride 128): I + codes * 2^e on the strict
// lower part, 0 above the diagonal
__device__ __forceinline__ void store_deq_diag(float* td, const AccI<4>& Tr, int e) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = 0; J < 4; ++J) {
      f32x4 x = zero4();
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int d = 16 * (I - J) + c - 4 * g - v;
        if (J <= I && d > 0) x[v] = ldexpf((float)Tr.a[bidx(I, J)][v], e);
        if (d == 0) x[v] = 1.f;
      }
      *(f32x4*)(td + (I * 16 + c) * 128 + J * 16 + 4 * g) = x;
    }
}

// LDS hand-over of 64 x 64 matrices of codes (|code| <= 32639) as int16 in
// padded rows of 72 (8-byte aligned runs of four, fewer bank conflicts on
// transposed access)
constexpr int kLD = 72;

__device__ __forceinline__ void lds_put4(short* p, i32x4 q) {
  *(int2*)p = int2{(int)((uint32_t)(q[0] & 0xffff) | ((uint32_t)q[1] << 16)),
                   (int)((uint32_t)(q[2] & 0xffff) | ((uint32_t)q[3] << 16))};
}
__device__ __forceinline__ i32x4 lds_get4(const short* p) {
  const int2 w = *(const int2*)p;
  return i32x4{(int)(int16_t)(w.x & 0xffff), w.x >> 16, (int)(int16_t)(w.y & 0xffff), w.y >> 16};
}

// LDS of one C = 128 tile: N11 (transposed), N22 and A21 (row-major), the
// exponents and flags, and the two maxima exchanged by the merge.
struct Lds128 {
  short n11t[64 * kLD];  // n11t[j * kLD + i] = N11[i][j]
  short n22[64 * kLD];
  short a21[64 * kLD];
  int info[20];  // e11, nz11, ea, e22, nz22, -, max P (2 waves), -, max X21 (2 waves), -,
                 // magnitudes of P's terms (2 x 2 waves), of X21's terms (2 x 2 waves)
};

// Wave 0 parks the codes of A21 (row form, all 16 blocks) and their
// exponent in LDS, before its engine runs (read after the workgroup barrier
// of int128_tile).
__device__ __forceinline__ void stash_a21(const FullI& A, int ea, Lds128& sh) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = 0; J < 4; ++J) lds_put4(&sh.a21[(16 * I + c) * kLD + 16 * J + 4 * g], A.a[4 * I + J]);
  if (lane_id() == 0) sh.info[2] = ea;
}

// The block columns J0 .. J0 + JN - 1 of out = q(t1 2^e1 + t2 2^e2): t1
// the codes of the row-form fragments X, t2 the exact product D.  The sum
// is exact in fp64 (both terms aligned at the finer exponent) under the
// exponent plan of sum_plan (intq.hpp); the terms' actual magnitudes are
// measured only when their bounds span more than 52 bits.  Every maximum is
// joined with the other wave's by join(m, slot) (slot s0 for the sum, s1,
// s2 for the terms' magnitudes), and the sum is quantised once by the
// scale rule.  The other block columns of out are set to 0.
template <typename W, int J0, int JN, typename Join>
__device__ __forceinline__ void sum2_full(FullI& out, int& eo, bool& nz, const typename W::Row& X,
                                          int e1, bool p1, const typename W::FProd& D, int e2,
                                          bool p2, Join&& join, int s0, int s1, int s2) {
  constexpr int Q = W::kQ, QB = W::kQB, ACCB = W::kAccB;
  int e[3] = {e1, e2, 0}, b[3] = {QB, ACCB, 0};
  bool p[3] = {p1, p2, false};
  if (p1 && p2 && max(e1 + QB, e2 + ACCB) - min(e1, e2) > 52) {
    int m1 = 0, m2 = 0;
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int K = J0; K < J0 + JN; ++K) {
        const i32x4 c1 = W::codes(X, I, K);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          m1 = max(m1, __double2hiint(fabs((double)c1[v])));
          m2 = max(m2, __double2hiint(fabs(elem(D.a[4 * I + K], v))));
        }
      }
    m1 = join(wave_max(m1), s1);
    m2 = join(wave_max(m2), s2);
    int q1 = 0, q2 = 0;
    if (m1) frexp(__hiloint2double(m1, 0), &q1);
    if (m2) frexp(__hiloint2double(m2, 0), &q2);
    b[0] = q1;
    b[1] = q2;
    p[0] = m1 > 0;
    p[1] = m2 > 0;
  }
  const SumPlan pl = (p[0] || p[1]) ? sum_plan<QB>(e, b, p) : SumPlan{0, {false, false, false},
                                                                        {false, false, false}};
  const double sa = pl.p[0] ? ldexp(1.0, e1 - pl.emin) : 0.0;
  const double sb = pl.p[1] ? ldexp(1.0, e2 - pl.emin) : 0.0;
  auto val = [&](int I, int K, int v, i32x4 c1) {
    double x = 0.0;
    if (pl.p[0]) {
      const double t = (double)c1[v] * sa;
      x += pl.r[0] ? rint(t) : t;
    }
    if (pl.p[1]) {
      const double t = elem(D.a[4 * I + K], v) * sb;
      x += pl.r[1] ? rint(t) : t;
    }
    return x;
  };
  int mh = 0;
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int K = J0; K < J0 + JN; ++K) {
      const i32x4 c1 = W::codes(X, I, K);
#pragma unroll
      for (int v = 0; v < 4; ++v) mh = max(mh, __double2hiint(fabs(val(I, K, v, c1))));
    }
  const int amax_hi = join(wave_max(mh), s0);
  nz = amax_hi > 0;
  const int s = nz ? shift_canon_hi<Q, QB>(amax_hi) : 0;
  const double sc = ldexp(1.0, -s);
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int K = 0; K < 4; ++K) {
      i32x4 r = zero_i4();
      if (nz && K >= J0 && K < J0 + JN) {
        const i32x4 c1 = W::codes(X, I, K);
#pragma unroll
        for (int v = 0; v < 4; ++v) r[v] = rne_scaled(val(I, K, v, c1), sc);
      }
      out.a[4 * I + K] = r;
    }
  eo = nz ? pl.emin + s : 0;
}

// Wave w's half of X21 = -(X22 (A21 X11)): the output block columns
// J0, J0 + 1 (J0 = 2 w) of P = A21 + A21 N11 and of X21 = -(P + N22 P).
// Column J of P needs all of A21 and column J of N11; column J of X21 needs
// all of N22 and column J of P; only the requantisation of each (one
// exponent per matrix) needs the other wave: its maximum, through LDS.
template <typename W, int J0>
__device__ __forceinline__ void merge_half(const AccI<4>& Tr, int eTo, bool nzT, Lds128& sh,
                                          typename W::Code* __restrict__ t,
                                          int32_t* __restrict__ et, float* __restrict__ td) {
  constexpr int C = 128, LD = kLD, wv = J0 / 2;
  const int g = lane_g(), c = lane_c();
  // the other wave's maximum joined with this wave's (wave-uniform values)
  auto xmax = [&](int m, int slot) {
    if (lane_id() == 0) sh.info[slot + wv] = m;
    __syncthreads();
    return max(__builtin_amdgcn_readfirstlane(sh.info[slot]),
               __builtin_amdgcn_readfirstlane(sh.info[slot + 1]));
  };
  const int e11 = __builtin_amdgcn_readfirstlane(sh.info[0]);
  const bool nz11 = __builtin_amdgcn_readfirstlane(sh.info[1]) != 0;
  const int ea = __builtin_amdgcn_readfirstlane(sh.info[2]);
  const int e22 = __builtin_amdgcn_readfirstlane(sh.info[3]);
  const bool nz22 = __builtin_amdgcn_readfirstlane(sh.info[4]) != 0;

  // column form of N11's block columns J0, J0 + 1 (lane (g, c) holds rows
  // 16 K + 4 g + v of column 16 J + c); the other columns are not used
  AccI<4> N11c;
#pragma unroll
  for (int J = 0; J < 4; ++J)
#pragma unroll
    for (int K = J; K < 4; ++K)
      N11c.a[bidx(K, J)] = (J >= J0 && J < J0 + 2)
                               ? lds_get4(&sh.n11t[(16 * J + c) * LD + 16 * K + 4 * g])
                               : zero_i4();
  typename W::Col N11q;
  W::to_col(N11q, N11c, 1, 63);
  FullI A21;
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = 0; J < 4; ++J) A21.a[4 * I + J] = lds_get4(&sh.a21[(16 * I + c) * LD + 16 * J + 4 * g]);
  const bool nzA = amax_full(A21) > 0;

  typename W::Row X;  // A21, then P, as row-form fragments (sum2_full reads the codes back)
  typename W::FProd D;
  W::to_frow(X, A21);
  W::template fmm<true, J0, 2>(D, X, N11q);  // A21 N11, row form, own columns
  FullI P;
  int eP;
  bool nzP;
  sum2_full<W, J0, 2>(P, eP, nzP, X, ea, nzA, D, ea + e11, nzA && nz11, xmax, 6, 12, 14);

  RowQ<4> Iq;
  ColQ<4> Ic;
  eye_quads(Iq, Ic);
  W::to_frow(X, P);  // P's other block columns are 0
  typename W::Col Pc;
  W::frow_to_col(Pc, X, Ic);
  typename W::Row N22q;
  if constexpr (J0 == 2) {
    W::to_row(N22q, Tr, 1, 63);
  } else {
    AccI<4> N22;
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) N22.a[bidx(I, J)] = lds_get4(&sh.n22[(16 * I + c) * LD + 16 * J + 4 * g]);
    W::to_row(N22q, N22, 1, 63);
  }
  W::template fmm<true, J0, 2>(D, N22q, Pc);  // N22 P, row form, own columns
  FullI Xs;
  int e21;
  bool nz21;
  sum2_full<W, J0, 2>(Xs, e21, nz21, X, eP, nzP, D, e22 + eP, nz22 && nzP, xmax, 9, 16, 18);

#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = J0; J < J0 + 2; ++J)
      W::store4(t + (64 + I * 16 + c) * C + J * 16 + 4 * g, zero_i4() - Xs.a[4 * I + J]);
  if (J0 == 2 && lane_id() == 0) et[1] = e21;
  if (td)
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = J0; J < J0 + 2; ++J) {
        f32x4 x;
#pragma unroll
        for (int v = 0; v < 4; ++v) x[v] = ldexpf((float)-Xs.a[4 * I + J][v], e21);
        *(f32x4*)(td + (64 + I * 16 + c) * C + J * 16 + 4 * g) = x;
      }
}

// One C = 128 tile after the diagonal blocks' codes are in registers (and,
// from wave 0, A21 in LDS by stash_a21).  Wave w (w = 0, 1) holds
// Lm = -A_ww (row form, strict lower) with exponent eL; it inverts its block
// with the engine and writes it, hands it to the other wave through LDS, and
// forms its half of X21 (merge_half).  Outputs for the tile: t (codes,
// 128 x 128), et (three exponents), td (nullable, fp32).
template <typename W, int NC, int SC>
__device__ __forceinline__ void int128_tile(int wv, const AccI<4>& Lr, int eL,
                                            typename W::Code* __restrict__ t,
                                            int32_t* __restrict__ et, float* __restrict__ td,
                                            int Nrt, int Srt, Lds128& sh) {
  constexpr int C = 128, LD = kLD;
  const int g = lane_g(), c = lane_c();
  const int r0 = 64 * wv;
  AccI<4> Tr;
  int eTo;
  W::template engine<NC, SC>(Lr, eL, Nrt, Srt, Tr, eTo);

  // ---- the diagonal block out (wave 0 also writes block 12, all zero)
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = 0; J < 4; ++J)
      W::store4(t + (r0 + I * 16 + c) * C + r0 + J * 16 + 4 * g,
                J <= I ? Tr.a[bidx(I, J)] : zero_i4());
  if (wv == 0)
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J < 4; ++J) W::store4(t + (I * 16 + c) * C + 64 + J * 16 + 4 * g, zero_i4());
  if (lane_id() == 0) et[2 * wv] = eTo;
  if (td) {
    store_deq_diag(td + r0 * C + r0, Tr, eTo);
    if (wv == 0)
#pragma unroll
      for (int I = 0; I < 4; ++I)
#pragma unroll
        for (int J = 0; J < 4; ++J) *(f32x4*)(td + (I * 16 + c) * C + 64 + J * 16 + 4 * g) = zero4();
  }
  const bool nzT = amax_of(Tr, 1, 63) > 0;
  if (wv == 0) {
    // N11 (row form: lane (g, c) holds row 16 I + c, columns 16 J + 4 g + v)
    // to LDS transposed, so that its column form reads as runs of four
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          sh.n11t[(16 * J + 4 * g + v) * LD + 16 * I + c] = (short)Tr.a[bidx(I, J)][v];
    if (lane_id() == 0) {
      sh.info[0] = eTo;
      sh.info[1] = nzT ? 1 : 0;
    }
  } else {
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) lds_put4(&sh.n22[(16 * I + c) * LD + 16 * J + 4 * g], Tr.a[bidx(I, J)]);
    if (lane_id() == 0) {
      sh.info[3] = eTo;
      sh.info[4] = nzT ? 1 : 0;
    }
  }
  __syncthreads();
  if (wv == 0)
    merge_half<W, 0>(Tr, eTo, nzT, sh, t, et, td);
  else
    merge_half<W, 2>(Tr, eTo, nzT, sh, t, et, td);
}

// The integer inverse at C = 128 from codes (gdn_quantize_tiles_* layout).
// Both C = 128 kernels are held to two waves per SIMD (amdgpu_waves_per_eu):
// INT8 then fits its registers exactly, INT16 keeps about 125 values in
// scratch memory; measured on 16384 tiles, 11-31 % less time than at one
// wave per SIMD.
template <typename W, int NC, int SC>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2)))
void k_neumann_int128(const typename W::Code* __restrict__ Aq,
                                                        const int32_t* __restrict__ eA,
                                                        typename W::Code* __restrict__ Tq,
                                                        int32_t* __restrict__ eT,
                                                        float* __restrict__ Tdeq, int Nrt,
                                                        int Srt) {
  using Code = typename W::Code;
  constexpr int C = 128;
  __shared__ __attribute__((aligned(16))) Lds128 sh;
  const int64_t tile = blockIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane_g(), c = lane_c();
  const int r0 = 64 * wv;
  const Code* a = Aq + tile * (C * C);

  // ---- this wave's diagonal block: Lm = -A_ww (row form), strictly lower
  AccI<4> Lr;
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      i32x4 x = W::load4(a + (r0 + I * 16 + c) * C + r0 + J * 16 + 4 * g);
#pragma unroll
      for (int v = 0; v < 4; ++v) x[v] = drow(I - J, v) > 0 ? -x[v] : 0;
      Lr.a[bidx(I, J)] = x;
    }
  const int eL = __builtin_amdgcn_readfirstlane(eA[3 * tile + 2 * wv]);
  if (wv == 0) {
    FullI A;
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J < 4; ++J) A.a[4 * I + J] = W::load4(a + (64 + I * 16 + c) * C + J * 16 + 4 * g);
    stash_a21(A, __builtin_amdgcn_readfirstlane(eA[3 * tile + 1]), sh);
  }
  int128_tile<W, NC, SC>(wv, Lr, eL, Tq + tile * (C * C), eT + 3 * tile,
                         Tdeq ? Tdeq + tile * (C * C) : nullptr, Nrt, Srt, sh);
}

// The whole integer path at C = 128 in one launch: A in fp32 from K, beta,
// g (the values gdn_build_A writes: the same Gram products in the same order
// and the same gates), each block quantised in registers by the block-wise
// quantiser's rule, then the block-wise integer inverse.  Wave w forms its
// diagonal block; wave 0 also forms A21, before its engine.
template <typename W, int DK, typename F, typename TK, int NC, int SC>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2)))
void k_inverse_int128_fused(const TK* __restrict__ K,
                                                              const float* __restrict__ beta,
                                                              const float* __restrict__ g,
                                                              typename W::Code* __restrict__ Tq,
                                                              int32_t* __restrict__ eT,
                                                              float* __restrict__ Tdeq, int L,
                                                              int H, int Nrt, int Srt) {
  constexpr int C = 128;
  __shared__ float sb[C], sg[C];
  __shared__ __attribute__((aligned(16))) Lds128 sh;
  const Chunk ch = Chunk::by_rows(blockIdx.x, gridDim.x, L, H, C);
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const Lane ln = lane_here();
  const int64_t ldk = (int64_t)H * DK;
  {
    const int r = threadIdx.x;  // 128 threads, one row each
    const int64_t o = ((int64_t)ch.b * L + ch.t0 + r) * H + ch.h;
    sb[r] = beta[o];
    sg[r] = g[o];
  }
  __syncthreads();

  // ---- this wave's diagonal block of A (fp32, row form), quantised
  AccI<4> Lr;
  int eL;
  {
    Acc<4> G;
    {
      Pair<F> kp[4][DK / 32];
      load_rows<4, DK>(kp, K + ch.row(64 * wv, L, H, DK), ldk);
      gram_lower<4, DK, true>(G, kp);
    }
    gate_scale<4, true>(G, sb + 64 * wv, sg + 64 * wv, 1.f);
    float m = 0.f;
#pragma unroll
    for (int b = 0; b < nlower(4); ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) m = fmaxf(m, fabsf(G.a[b][v]));
    eL = W::qexp(
        __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(__ockl_wfred_max_f32(m)))));
#pragma unroll
    for (int b = 0; b < nlower(4); ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) Lr.a[b][v] = -(int)rintf(ldexpf(G.a[b][v], -eL));
  }
  // ---- A21 (wave 0, before its engine): the Gram of the K rows of half 2
  // against those of half 1, slice by slice in the feature order of the
  // full Gram product, then the gates, then its own exponent
  if (wv == 0) {
    f32x4 G2[4][4];
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J < 4; ++J) G2[I][J] = zero4();
#pragma unroll
    for (int q = 0; q < DK / 32; ++q) {
      Pair<F> k1[4], k2[4];
#pragma unroll
      for (int I = 0; I < 4; ++I) {
        k1[I] = load_row8<F>(K + ch.row(I * 16 + ln.c(), L, H, DK) + 32 * q + 8 * ln.g());
        k2[I] = load_row8<F>(K + ch.row(64 + I * 16 + ln.c(), L, H, DK) + 32 * q + 8 * ln.g());
      }
#pragma unroll
      for (int I = 0; I < 4; ++I)
#pragma unroll
        for (int J = 0; J < 4; ++J) G2[I][J] = Pair<F>::template mma<true>(k2[I], k1[J], G2[I][J]);
    }
    const int gg = ln.g(), c = ln.c();
    float m = 0.f;
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J < 4; ++J)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int i = 64 + I * 16 + c, j = J * 16 + 4 * gg + v;
          G2[I][J][v] = 1.f * sb[i] * G2[I][J][v] * __expf(sg[i] - sg[j]);
          m = fmaxf(m, fabsf(G2[I][J][v]));
        }
    const int ea = W::qexp(
        __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(__ockl_wfred_max_f32(m)))));
    FullI A;
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J < 4; ++J)
#pragma unroll
        for (int v = 0; v < 4; ++v) A.a[4 * I + J][v] = (int)rintf(ldexpf(G2[I][J][v], -ea));
    stash_a21(A, ea, sh);
  }
  int128_tile<W, NC, SC>(wv, Lr, eL, Tq + ch.tile * (C * C), eT + 3 * ch.tile,
                         Tdeq ? Tdeq + ch.tile * (C * C) : nullptr, Nrt, Srt, sh);
}

// Quantiser at C = 128: four waves per tile, wave w on the 64 x 64 quadrant
// (w >> 1, w & 1).  The strict lower parts of the diagonal blocks and the
// whole block 21 each get their own exponent (the per-tile rule applied to
// the block: codes round-half-even(x / 2^e), e the smallest integer at which
// they lie in [-qmax, qmax]); block 12 is written as 0.  eA[3 tile + k] for
// the blocks k = 0 (11), 1 (21), 2 (22).
template <typename W>
__global__ __launch_bounds__(256) void k_quantize_int128(const float* __restrict__ A,
                                                         typename W::Code* __restrict__ Aq,
                                                         int32_t* __restrict__ eA) {
  constexpr int C = 128, PER = 16;  // float4 per lane of a 64 x 64 block
  const int64_t tile = blockIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int qr = wv >> 1, qc = wv & 1;
  const int l = lane_id();
  typename W::Code* q = Aq + tile * (C * C) + (64 * qr) * C + 64 * qc;
  if (qr == 0 && qc == 1) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = k * 64 + l;
      W::store4(q + (idx >> 4) * C + (idx & 15) * 4, zero_i4());
    }
    return;
  }
  const float* a = A + tile * (C * C) + (64 * qr) * C + 64 * qc;
  f32x4 x[PER];
  float m = 0.f;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int idx = k * 64 + l;
    const int row = idx >> 4, col = (idx & 15) * 4;
    x[k] = *(const f32x4*)(a + row * C + col);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if (qr == qc && row <= col + v) x[k][v] = 0.f;
      m = fmaxf(m, fabsf(x[k][v]));
    }
  }
  const float amax =
      __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(__ockl_wfred_max_f32(m))));
  const int e = W::qexp(amax);
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int idx = k * 64 + l;
    i32x4 r;
#pragma unroll
    for (int v = 0; v < 4; ++v) r[v] = (int)rintf(ldexpf(x[k][v], -e));
    W::store4(q + (idx >> 4) * C + (idx & 15) * 4, r);
  }
  if (l == 0) eA[3 * tile + qr + qc] = e;
}

}  // namespace iq
}  // namespace gdn
