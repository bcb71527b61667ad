// neumann.hip -- standalone MatMul-only chunk inverse (one wave per tile).
//
// C in {16, 32, 64}: the whole tile is one register-resident engine
// (engine.hpp).  C = 128: block-wise (Appendix E, Appendix H of
// arXiv 2606.06034): both 64 x 64 diagonal blocks through the engine, joined
// by T_21 = -T_22 A_21 T_11.
#include "engine.hpp"
#include "launch.hpp"

namespace gdn {

template <int NB, typename F, typename TIO>
__global__ __launch_bounds__(64) void k_neumann(const TIO* __restrict__ A, TIO* __restrict__ T,
                                                int N, int S) {
  constexpr int C = 16 * NB, NL = nlower(NB);
  const int64_t tile = blockIdx.x;
  const TIO* a = A + tile * (C * C);
  TIO* t = T + tile * (C * C);
  F LQ[NL], LC[NL];
  load_neg_strict_row<NB>(a, C, LQ);
  {
    f32x4 tmp[NL];
    to_col<NB>(tmp, LQ, 1, C - 1);
    cvt_all<NB>(LC, tmp);
  }
  f32x4 Tr[NL];
  neumann_engine<NB>(LQ, LC, N, S, Tr);
  store_unit_row<NB>(t, C, Tr);
}

// ---------------------------------------------------------------------------
// C = 128 as 2 x 2 blocks of 64 (four 16-blocks each)

template <typename F, typename TIO>
__global__ __launch_bounds__(64) void k_neumann128(const TIO* __restrict__ A,
                                                   TIO* __restrict__ T, int N, int S) {
  constexpr int C = 128, NB = 4, NL = nlower(NB);
  const int64_t tile = blockIdx.x;
  const TIO* a = A + tile * (C * C);
  TIO* t = T + tile * (C * C);
  const int g = lane_g(), c = lane_c();

  // T_22 first; keep it (unit lower, row form) as an operand.
  F X22r[NL];
  {
    F LQ[NL], LC[NL];
    load_neg_strict_row<NB>(a + 64 * C + 64, C, LQ);
    f32x4 tmp[NL];
    to_col<NB>(tmp, LQ, 1, 63);
    cvt_all<NB>(LC, tmp);
    f32x4 Tr[NL];
    neumann_engine<NB>(LQ, LC, N, S, Tr);
    store_unit_row<NB>(t + 64 * C + 64, C, Tr);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) {
        f32x4 x = Tr[bidx(I, J)];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int d = dQ(I, J, v);
          x[v] = d > 0 ? x[v] : (d == 0 ? 1.f : 0.f);
        }
        X22r[bidx(I, J)] = Op<F>::from(x);
      }
  }

  // T_11, as a column-form operand (right factor of A_21 T_11)
  F X11c[NL];
  {
    F LQ[NL], LC[NL];
    load_neg_strict_row<NB>(a, C, LQ);
    f32x4 tmp[NL];
    to_col<NB>(tmp, LQ, 1, 63);
    cvt_all<NB>(LC, tmp);
    f32x4 Tr[NL];
    neumann_engine<NB>(LQ, LC, N, S, Tr);
    store_unit_row<NB>(t, C, Tr);
    F X11r[NL];
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J) {
        f32x4 x = Tr[bidx(I, J)];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int d = dQ(I, J, v);
          x[v] = d > 0 ? x[v] : (d == 0 ? 1.f : 0.f);
        }
        X11r[bidx(I, J)] = Op<F>::from(x);
      }
    to_col<NB>(tmp, X11r, 0, 63);
    cvt_all<NB>(X11c, tmp);
  }
  // upper-right 64 x 64 block of the tile is zero
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J) store4(t + (I * 16 + c) * C + 64 + J * 16 + 4 * g, zero4());

  // M = A_21 T_11 (dense 64 x 64, column form)
  F Mc[NB * NB];
  {
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      F a21[NB];
#pragma unroll
      for (int K = 0; K < NB; ++K)
        a21[K] = Op<F>::from(load4(a + (64 + I * 16 + c) * C + K * 16 + 4 * g));
#pragma unroll
      for (int J = 0; J < NB; ++J) {
        f32x4 acc = zero4();
#pragma unroll
        for (int K = J; K < NB; K += 2) {
          if (K + 1 < NB)
            acc = Op<F>::template pair<false>(a21[K], a21[K + 1], X11c[bidx(K, J)],
                                              X11c[bidx(K + 1, J)], acc);
          else
            acc = Op<F>::template one<false>(a21[K], X11c[bidx(K, J)], acc);
        }
        Mc[I * NB + J] = Op<F>::from(acc);
      }
    }
  }
  // T_21 = -T_22 M (row form), stored
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J) {
      f32x4 acc = zero4();
#pragma unroll
      for (int K = 0; K <= I; K += 2) {
        if (K + 1 <= I)
          acc = Op<F>::template pair<true>(X22r[bidx(I, K)], X22r[bidx(I, K + 1)],
                                           Mc[K * NB + J], Mc[(K + 1) * NB + J], acc);
        else
          acc = Op<F>::template one<true>(X22r[bidx(I, K)], Mc[K * NB + J], acc);
      }
      store4(t + (64 + I * 16 + c) * C + J * 16 + 4 * g, -acc);
    }
}

// ---------------------------------------------------------------------------

template <int NB, typename F, typename TIO>
static hipError_t run_neumann(const void* A, void* T, int64_t n, int N, int S, hipStream_t st) {
  hipLaunchKernelGGL((k_neumann<NB, F, TIO>), dim3((unsigned)n), dim3(64), 0, st,
                     (const TIO*)A, (TIO*)T, N, S);
  return hipGetLastError();
}

template <typename F, typename TIO>
static hipError_t run_neumann_c(const void* A, void* T, int64_t n, int C, int N, int S,
                                hipStream_t st) {
  switch (C) {
    case 16: return run_neumann<1, F, TIO>(A, T, n, N, S, st);
    case 32: return run_neumann<2, F, TIO>(A, T, n, N, S, st);
    case 64: return run_neumann<4, F, TIO>(A, T, n, N, S, st);
    case 128:
      hipLaunchKernelGGL((k_neumann128<F, TIO>), dim3((unsigned)n), dim3(64), 0, st,
                         (const TIO*)A, (TIO*)T, N, S);
      return hipGetLastError();
  }
  return hipErrorNotSupported;
}

hipError_t launch_neumann(const void* A, void* T, int64_t n, int C, int N, int S, int dtype,
                          hipStream_t st) {
  if (dtype == 0) return run_neumann_c<f32x4, float>(A, T, n, C, N, S, st);
  if (dtype == 1) return run_neumann_c<bf16x4, __bf16>(A, T, n, C, N, S, st);
  return hipErrorNotSupported;
}

}  // namespace gdn
