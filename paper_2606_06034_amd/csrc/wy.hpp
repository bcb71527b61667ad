// wy.hpp -- applying a chunk's inverse to token-major operands (WY form)
// and the shared front half of the fused kernels (A from K, then the
// inverse), used by the chunk pipeline and the layer forward.
//
//   W = T diag(beta) K,  U = T diag(beta) V          (Section 2.1)
//
// K/V rows of a chunk are strided by H * d in the [B, L, H, d] layout; every
// global access is a run of 8 consecutive features of one token (16 bytes in
// bf16).  Column-form (token-major) fragments of K and V are made on chip by
// identity MFMAs.
#pragma once

#include "chunk.hpp"
#include "engine.hpp"

namespace gdn {

// Asynchronous copy of a bf16 chunk of X into LDS (global -> LDS DMA, no
// registers): the 16-byte run lane (g, c) would load in load_rows lands at
// s + 512 (I * D / 32 + q) + 8 * lane.  Completion is tracked by vmcnt.
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;

// Rows r >= m are copied from row m - 1 (finite values that the zero
// columns of T diag(beta) cancel).
template <int NB, int D>
__device__ __forceinline__ void prefetch_rows_lds(const __bf16* __restrict__ xb, int64_t ld,
                                                  __bf16* s, Lane ln = lane_here(),
                                                  int m = 16 * NB) {
  const int g = ln.g(), c = ln.c();
#pragma unroll
  for (int I = 0; I < NB; ++I) {
    const int r = I * 16 + c, rr = r < m ? r : m - 1;
#pragma unroll
    for (int q = 0; q < D / 32; ++q)
      __builtin_amdgcn_global_load_lds((glb_void*)(xb + rr * ld + 32 * q + 8 * g),
                                       (lds_void*)(s + 512 * (I * (D / 32) + q)), 16, 0, 0);
  }
}

// wait for every outstanding vector-memory operation of this wave
// (s_waitcnt vmcnt(0))
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// out = T' X for one chunk, T' = T diag(beta) as row pairs (beta folded into
// T's columns), X given by get(I, q): its row-form pair of rows 16I..16I+15,
// features 32q..32q+31 (registers, or LDS read one 32-feature slice at a
// time).  Each 16 x 16 block of X is moved to column form by an identity
// MFMA (X I), then W(I, .) = sum_K T'(I, K) X(K, .) comes out in row form and
// is stored 8 features per lane.  ob points at (token t0, head h, feature 0)
// of the output; lds_copy (optional) receives the output pairs in the slot
// layout LdsRows reads.
template <int NB, int D, typename F, typename TIO, typename Get>
__device__ __forceinline__ void apply_lower(const RowP<NB, F>& TR, Get&& get,
                                            TIO* __restrict__ ob, int64_t ld,
                                            Lane ln = lane_here(), TIO* lds_copy = nullptr,
                                            int m = 16 * NB) {
  const int g = ln.g(), c = ln.c();
  const f32x4 e = eye4(ln);
  const Pair<F> id0 = Pair<F>::make(e, zero4()), id1 = Pair<F>::make(zero4(), e);
#pragma unroll
  for (int q = 0; q < D / 32; ++q) {
    Pair<F> x[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) x[I] = get(I, q);
    Pair<F> y[2][npair(NB)];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int p = 0; p < npair(NB); ++p) {
        const f32x4 a = Pair<F>::template mma<false>(x[2 * p], h ? id1 : id0, zero4());
        const f32x4 b = (2 * p + 1 < NB)
                            ? Pair<F>::template mma<false>(x[2 * p + 1], h ? id1 : id0, zero4())
                            : zero4();
        y[h][p] = Pair<F>::make(a, b);
      }
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      f32x4 acc[2] = {zero4(), zero4()};
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int p = 0; p < npair(NB); ++p)
          if (2 * p <= I) acc[h] = Pair<F>::template mma<true>(TR.r[I][p], y[h][p], acc[h]);
      if (I * 16 + c < m) store_row8(ob + (I * 16 + c) * ld + 32 * q + 8 * g, acc[0], acc[1]);
      if (lds_copy) store_row8(lds_copy + 512 * (I * (D / 32) + q) + 8 * ln.id, acc[0], acc[1]);
    }
  }
}
// operand getters: pairs held in registers, or the LDS copy prefetch_rows_lds
// made (one 16-byte read per lane and pair)
template <int NB, int D, typename F>
struct RegRows {
  const Pair<F> (&xp)[NB][D / 32];
  __device__ __forceinline__ Pair<F> operator()(int I, int q) const { return xp[I][q]; }
};
// slot (I, q) of an LDS copy: 8 elements per lane, lane-major
template <int D, typename F = bf16x4, typename TIO = __bf16>
struct LdsRows {
  const TIO* s;
  int l;
  __device__ __forceinline__ Pair<F> operator()(int I, int q) const {
    return load_row8<F>(s + 512 * (I * (D / 32) + q) + 8 * l);
  }
};

// T diag(beta) as row pairs from the row-form blocks of the unit lower T:
// value v of lane (g, c) in block (I, J) sits in column 16J + 4g + v.
template <int NB, typename F>
__device__ __forceinline__ void scale_cols(RowP<NB, F>& TR, Acc<NB> T, const float* sb,
                                           Lane ln = lane_here()) {
  const int g = ln.g();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
#pragma unroll
      for (int v = 0; v < 4; ++v) T.a[bidx(I, J)][v] *= sb[16 * J + 4 * g + v];
  to_rowp(TR, T);
}

// The inverse of (I + A) for one chunk from its K row pairs, in row form
// with the unit diagonal included: T_hat(N, S) by the engine, or (EXACT)
// the exact block-wise inverse.  `after_gram` runs right after the Gram
// product (the fused kernels start DMA copies there).
template <int NB, int DK, typename F, bool SMALLN, int NC, int SC, bool EXACT, typename Hook>
__device__ __forceinline__ void chunk_inverse(const Pair<F> (&kp)[NB][DK / 32], const float* sb,
                                              const float* sg, int N, int S, Acc<NB>& Tr,
                                              Hook&& after_gram) {
  constexpr int C = 16 * NB;
  if constexpr (EXACT) {
    Acc<NB> Lr;
    gram_lower<NB, DK, true>(Lr, kp);
    after_gram();
    gate_scale<NB, true>(Lr, sb, sg, -1.f);  // Lm = -A, row form
    blockwise_inverse<NB, F>(Lr, Tr);
  } else {
    RowP<NB, F> LR;
    Acc<NB> Lc;
    {
      gram_lower<NB, DK, false>(Lc, kp);
      after_gram();
      gate_scale<NB, false>(Lc, sb, sg, -1.f);  // Lm = -A, column form
      ColP<NB, F> LC;
      to_colp(LC, Lc);
      Acc<NB> r;
      col_to_row(r, LC, 1, C - 1);
      to_rowp(LR, r);
    }
    neumann_engine<NB, F, SMALLN, NC, SC>(LR, Lc, N, S, Tr);
  }
}

}  // namespace gdn
