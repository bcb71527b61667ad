// neumann.hip -- standalone MatMul-only chunk inverse (one wave per tile).
//
// C in {16, 32, 64}: the whole tile is one register-resident engine
// (engine.hpp).  C = 128: block-wise (Appendix E, Appendix H of
// arXiv 2606.06034): both 64 x 64 diagonal blocks through the engine, joined
// by T_21 = -T_22 A_21 T_11.
#include "engine.hpp"
#include "launch.hpp"

namespace gdn {

// GH selects the residual sum's evaluation (engine.hpp): Horner for the
// standalone tiles, the power chain inside the C = 128 kernel (measured
// faster there, where the merge adds to the register load).  EXACT: the
// exact block-wise inverse instead of T_hat(N, S).
// the inverse of a tile whose lower-triangle blocks R are already loaded
template <int NB, typename F, bool SMALLN, int NC, int SC, bool GH = true, bool EXACT = false>
__device__ __forceinline__ void invert_loaded(const Acc<NB>& R, int N, int S, Acc<NB>& Tr) {
  if constexpr (EXACT) {
    Acc<NB> Lr;
    neg_strict_row_from<NB>(R, Lr);
    blockwise_inverse<NB, F>(Lr, Tr);
  } else {
    Acc<NB> Lr, Lc;
    neg_strict_from<NB, F, SMALLN>(R, NC >= 0 ? NC : N, Lr, Lc);
    RowP<NB, F> LR;
    to_rowp(LR, Lr);
    neumann_engine<NB, F, SMALLN, NC, SC, GH>(LR, Lc, N, S, Tr);
  }
}

template <int NB, typename F, bool SMALLN, int NC, int SC, typename TIO, bool GH = true,
          bool EXACT = false>
__device__ __forceinline__ void invert_block(const TIO* __restrict__ a, TIO* __restrict__ t,
                                             int ldr, int N, int S, Acc<NB>& Tr) {
  Acc<NB> R;
  load_lower_raw<NB>(a, ldr, R);
  invert_loaded<NB, F, SMALLN, NC, SC, GH, EXACT>(R, N, S, Tr);
  store_unit_row<NB>(t, ldr, Tr);
}

// Tiles per wave: at C = 16, 32 one tile moves only 4 or 8 elements per
// lane, too few bytes in flight to cover HBM latency; a wave then issues
// the loads of several tiles before it computes on the first.
template <int NB> struct TilesPerWave { static constexpr int W = NB == 1 ? 4 : NB == 2 ? 2 : 1; };
template <int NB> dim3 tile_grid(int64_t n) {
  return dim3((unsigned)((n + TilesPerWave<NB>::W - 1) / TilesPerWave<NB>::W));
}

template <int NB, typename F, bool SMALLN, int NC, int SC, typename TIO, bool EXACT = false>
__global__ __launch_bounds__(64) void k_neumann(const TIO* __restrict__ A, TIO* __restrict__ T,
                                                int64_t n, int N, int S) {
  constexpr int C = 16 * NB, W = TilesPerWave<NB>::W;
  const int64_t tile0 = (int64_t)blockIdx.x * W;
  Acc<NB> R[W];
#pragma unroll
  for (int w = 0; w < W; ++w)
    if (W == 1 || tile0 + w < n) load_lower_raw<NB>(A + (tile0 + w) * (C * C), C, R[w]);
#pragma unroll
  for (int w = 0; w < W; ++w)
    if (W == 1 || tile0 + w < n) {
      Acc<NB> Tr;
      invert_loaded<NB, F, SMALLN, NC, SC, true, EXACT>(R[w], N, S, Tr);
      store_unit_row<NB>(T + (tile0 + w) * (C * C), C, Tr);
    }
}

// ---------------------------------------------------------------------------
// C = 128 as 2 x 2 blocks of 64 (four 16-blocks each)

template <typename F, bool SMALLN, int NC, int SC, typename TIO, bool EXACT = false>
__global__ __launch_bounds__(64) void k_neumann128(const TIO* __restrict__ A,
                                                   TIO* __restrict__ T, int N, int S) {
  constexpr int C = 128, NB = 4;
  const int64_t tile = blockIdx.x;
  const TIO* a = A + tile * (C * C);
  TIO* t = T + tile * (C * C);
  const int g = lane_g(), c = lane_c();

  // T_22 (row pairs, unit diagonal): left factor of T_22 M
  RowP<NB, F> X22;
  {
    Acc<NB> Tr;
    invert_block<NB, F, SMALLN, NC, SC, TIO, false, EXACT>(a + 64 * C + 64, t + 64 * C + 64, C, N, S, Tr);
#pragma unroll
    for (int I = 0; I < NB; ++I) Tr.a[bidx(I, I)] = band_block<false>(Tr.a[bidx(I, I)], 0, 1, 64) + eye4();
    to_rowp(X22, Tr);
  }
  // T_11 (column pairs): right factor of A_21 T_11
  ColP<NB, F> X11;
  {
    Acc<NB> Tr, Tc;
    invert_block<NB, F, SMALLN, NC, SC, TIO, false, EXACT>(a, t, C, N, S, Tr);
#pragma unroll
    for (int I = 0; I < NB; ++I) Tr.a[bidx(I, I)] = band_block<false>(Tr.a[bidx(I, I)], 0, 1, 64) + eye4();
    RowP<NB, F> X11r;
    to_rowp(X11r, Tr);
    row_to_col(Tc, X11r, 0, 63);
    to_colp(X11, Tc);
  }
  // upper-right 64 x 64 block of the tile is zero
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J) store4(t + (I * 16 + c) * C + 64 + J * 16 + 4 * g, zero4());

  // M = A_21 T_11, dense 4 x 4 blocks, as column pairs of the next product
  Pair<F> Mp[npair(NB)][NB];
  {
    f32x4 M[NB][NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      Pair<F> ar[npair(NB)];
#pragma unroll
      for (int p = 0; p < npair(NB); ++p)
        ar[p] = Pair<F>::make(load4(a + (64 + I * 16 + c) * C + 32 * p + 4 * g),
                              load4(a + (64 + I * 16 + c) * C + 32 * p + 16 + 4 * g));
#pragma unroll
      for (int J = 0; J < NB; ++J) {
        f32x4 acc = zero4();
#pragma unroll
        for (int p = 0; p < npair(NB); ++p)
          if (2 * p + 1 >= J) acc = Pair<F>::template mma<false>(ar[p], X11.c[p][J], acc);
        M[I][J] = acc;
      }
    }
#pragma unroll
    for (int p = 0; p < npair(NB); ++p)
#pragma unroll
      for (int J = 0; J < NB; ++J) Mp[p][J] = Pair<F>::make(M[2 * p][J], M[2 * p + 1][J]);
  }
  // T_21 = -T_22 M (row form), stored
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J) {
      f32x4 acc = zero4();
#pragma unroll
      for (int p = 0; p < npair(NB); ++p)
        if (2 * p <= I) acc = Pair<F>::template mma<true>(X22.r[I][p], Mp[p][J], acc);
      store4(t + (64 + I * 16 + c) * C + J * 16 + 4 * g, -acc);
    }
}

// ---------------------------------------------------------------------------

// Default order of each chunk size (the table of gdn_default_order) runs a
// kernel with (N, S) fixed at compile time; any other order runs the
// runtime-order kernel.
template <int NB> struct DefaultOrder;
template <> struct DefaultOrder<1> { static constexpr int N = 3, S = 2; };
template <> struct DefaultOrder<2> { static constexpr int N = 3, S = 4; };
template <> struct DefaultOrder<4> { static constexpr int N = 3, S = 8; };

template <int NB, typename F, typename TIO>
static hipError_t run_neumann(const void* A, void* T, int64_t n, int N, int S, hipStream_t st) {
  constexpr int DN = DefaultOrder<NB>::N, DS = DefaultOrder<NB>::S;
  const dim3 grid = tile_grid<NB>(n), block(64);
  if (N == DN && S == DS)
    hipLaunchKernelGGL((k_neumann<NB, F, true, DN, DS, TIO>), grid, block, 0, st, (const TIO*)A,
                       (TIO*)T, n, N, S);
  else if (N <= 15)
    hipLaunchKernelGGL((k_neumann<NB, F, true, -1, -1, TIO>), grid, block, 0, st, (const TIO*)A,
                       (TIO*)T, n, N, S);
  else
    hipLaunchKernelGGL((k_neumann<NB, F, false, -1, -1, TIO>), grid, block, 0, st, (const TIO*)A,
                       (TIO*)T, n, N, S);
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
      if (N == 3 && S == 8)
        hipLaunchKernelGGL((k_neumann128<F, true, 3, 8, TIO>), dim3((unsigned)n), dim3(64), 0, st,
                           (const TIO*)A, (TIO*)T, N, S);
      else if (N <= 15)
        hipLaunchKernelGGL((k_neumann128<F, true, -1, -1, TIO>), dim3((unsigned)n), dim3(64), 0,
                           st, (const TIO*)A, (TIO*)T, N, S);
      else
        hipLaunchKernelGGL((k_neumann128<F, false, -1, -1, TIO>), dim3((unsigned)n), dim3(64),
                           0, st, (const TIO*)A, (TIO*)T, N, S);
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

// ---------------------------------------------------------------------------
// exact block-wise inverse (C <= 64 one engine call; C = 128 two 64-blocks and
// the merge above)

template <typename F, typename TIO>
static hipError_t run_blockwise(const void* A, void* T, int64_t n, int C, hipStream_t st) {
  const TIO* a = (const TIO*)A;
  TIO* t = (TIO*)T;
  switch (C) {
    case 16:
      hipLaunchKernelGGL((k_neumann<1, F, true, 0, 0, TIO, true>), tile_grid<1>(n), dim3(64), 0,
                         st, a, t, n, 0, 0);
      break;
    case 32:
      hipLaunchKernelGGL((k_neumann<2, F, true, 0, 0, TIO, true>), tile_grid<2>(n), dim3(64), 0,
                         st, a, t, n, 0, 0);
      break;
    case 64:
      hipLaunchKernelGGL((k_neumann<4, F, true, 0, 0, TIO, true>), tile_grid<4>(n), dim3(64), 0,
                         st, a, t, n, 0, 0);
      break;
    case 128:
      hipLaunchKernelGGL((k_neumann128<F, true, 0, 0, TIO, true>), dim3((unsigned)n), dim3(64), 0,
                         st, a, t, 0, 0);
      break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

hipError_t launch_blockwise(const void* A, void* T, int64_t n, int C, int dtype, hipStream_t st) {
  if (dtype == 0) return run_blockwise<f32x4, float>(A, T, n, C, st);
  if (dtype == 1) return run_blockwise<bf16x4, __bf16>(A, T, n, C, st);
  return hipErrorNotSupported;
}

}  // namespace gdn
