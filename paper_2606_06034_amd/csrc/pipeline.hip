// pipeline.hip -- building A, applying the inverse to K and V (WY form), and
// the fused chunk pipeline.  One wave per (batch, head, chunk) tile.
//
//   A_ij = beta_i (k_i . k_j) exp(g_i - g_j) for i > j       (Section 2.1)
//   W = T diag(beta) K,  U = T diag(beta) V
//
// K/V rows of a chunk are strided by H * d in the [B, L, H, d] layout; every
// access is a 4-element (8 or 16 byte) run of one token's features (row form)
// or a 16-lane run of one feature over consecutive lanes (column form).
#include "engine.hpp"
#include "launch.hpp"

namespace gdn {

__device__ __forceinline__ float ld1(const float* p) { return *p; }
__device__ __forceinline__ float ld1(const __bf16* p) { return (float)*p; }

// Chunk bookkeeping for tile index `tile` of the [B, H, L/C, C, C] layout.
struct Chunk {
  int b, h, t0;
  __device__ Chunk(int64_t tile, int L, int H, int C) {
    const int nc = L / C;
    const int64_t bh = tile / nc;
    t0 = (int)(tile - bh * nc) * C;
    b = (int)(bh / H);
    h = (int)(bh - (int64_t)b * H);
  }
  // element offset of (token t0 + r, head h, feature 0) in [B, L, H, d]
  __device__ int64_t row(int r, int L, int H, int d) const {
    return (((int64_t)b * L + t0 + r) * H + h) * d;
  }
};

// beta and g of the chunk into LDS (one wave; C <= 128)
template <int C>
__device__ __forceinline__ void load_gates(const float* __restrict__ beta,
                                           const float* __restrict__ g, const Chunk& ch, int L,
                                           int H, float* sb, float* sg) {
  for (int r = lane_id(); r < C; r += 64) {
    const int64_t o = ((int64_t)ch.b * L + ch.t0 + r) * H + ch.h;
    if (sb) sb[r] = beta[o];
    if (sg) sg[r] = g[o];
  }
  __syncthreads();
}

// Lower blocks of the chunk Gram matrix K K^T (fp32 accumulation).
// OUTQ selects the result form.  kb points at (token t0, head h, feature 0).
template <int NB, bool OUTQ, typename F, typename TK>
__device__ __forceinline__ void gram_lower(f32x4 (&G)[nlower(NB)], const TK* __restrict__ kb,
                                           int64_t ldk, int dk) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) G[b] = zero4();
  for (int f = 0; f < dk; f += 32) {
    F k0[NB], k1[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      const TK* p = kb + (I * 16 + c) * ldk + f + 4 * g;
      k0[I] = Op<F>::from(load4(p));
      k1[I] = Op<F>::from(load4(p + 16));
    }
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        G[bidx(I, J)] = Op<F>::template pair<OUTQ>(k0[I], k1[I], k0[J], k1[J], G[bidx(I, J)]);
  }
}

// A from the Gram blocks (in place): form-aware element coordinates.
template <int NB, bool ROWFORM>
__device__ __forceinline__ void gate_scale(f32x4 (&G)[nlower(NB)], const float* sb,
                                           const float* sg, float sign) {
  const int g = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = ROWFORM ? I * 16 + c : I * 16 + 4 * g + v;
        const int j = ROWFORM ? J * 16 + 4 * g + v : J * 16 + c;
        const float x = G[bidx(I, J)][v];
        G[bidx(I, J)][v] = (i > j) ? sign * sb[i] * x * __expf(sg[i] - sg[j]) : 0.f;
      }
}

// out = T diag(beta) X for one chunk.  Tq: unit lower T in row form;
// xb / ob point at (token t0, head h, feature 0) of X and of the output.
template <int NB, typename F, typename TIO>
__device__ __forceinline__ void apply_lower(const F (&Tq)[nlower(NB)], const TIO* __restrict__ xb,
                                            TIO* __restrict__ ob, int64_t ld, int d,
                                            const float* sb) {
  const int g = lane_g(), c = lane_c();
  for (int f = 0; f < d; f += 16) {
    F y[NB];
#pragma unroll
    for (int K = 0; K < NB; ++K) {
      f32x4 x;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int r = K * 16 + 4 * g + v;
        x[v] = sb[r] * ld1(xb + r * ld + f + c);
      }
      y[K] = Op<F>::from(x);
    }
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      f32x4 acc = zero4();
#pragma unroll
      for (int K = 0; K <= I; K += 2) {
        if (K + 1 <= I)
          acc = Op<F>::template pair<true>(Tq[bidx(I, K)], Tq[bidx(I, K + 1)], y[K], y[K + 1], acc);
        else
          acc = Op<F>::template one<true>(Tq[bidx(I, K)], y[K], acc);
      }
      store4(ob + (I * 16 + c) * ld + f + 4 * g, acc);
    }
  }
}

// ---------------------------------------------------------------------------
// gdn_build_A

template <int NB, typename F, typename TK, typename TA>
__global__ __launch_bounds__(64) void k_build_A(const TK* __restrict__ K,
                                                const float* __restrict__ beta,
                                                const float* __restrict__ g,
                                                TA* __restrict__ A, int L, int H, int dk) {
  constexpr int C = 16 * NB, NL = nlower(NB);
  __shared__ float sb[C], sg[C];
  const int64_t tile = blockIdx.x;
  const Chunk ch(tile, L, H, C);
  load_gates<C>(beta, g, ch, L, H, sb, sg);
  f32x4 G[NL];
  gram_lower<NB, true, F>(G, K + ch.row(0, L, H, dk), (int64_t)H * dk, dk);
  gate_scale<NB, true>(G, sb, sg, 1.f);
  TA* a = A + tile * (C * C);
  const int gg = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J)
      store4(a + (I * 16 + c) * C + J * 16 + 4 * gg, J <= I ? G[bidx(I, J)] : zero4());
}

// ---------------------------------------------------------------------------
// gdn_wy_apply

template <int NB, typename F, typename TIO>
__global__ __launch_bounds__(64) void k_wy(const TIO* __restrict__ T, const TIO* __restrict__ K,
                                           const TIO* __restrict__ V,
                                           const float* __restrict__ beta, TIO* __restrict__ W,
                                           TIO* __restrict__ U, int L, int H, int dk, int dv) {
  constexpr int C = 16 * NB, NL = nlower(NB);
  __shared__ float sb[C];
  const int64_t tile = blockIdx.x;
  const Chunk ch(tile, L, H, C);
  load_gates<C>(beta, beta, ch, L, H, sb, nullptr);
  const TIO* t = T + tile * (C * C);
  const int g = lane_g(), c = lane_c();
  F Tq[NL];
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 x = load4(t + (I * 16 + c) * C + J * 16 + 4 * g);
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (dQ(I, J, v) < 0) x[v] = 0.f;
      Tq[bidx(I, J)] = Op<F>::from(x);
    }
  apply_lower<NB>(Tq, K + ch.row(0, L, H, dk), W + ch.row(0, L, H, dk), (int64_t)H * dk, dk, sb);
  apply_lower<NB>(Tq, V + ch.row(0, L, H, dv), U + ch.row(0, L, H, dv), (int64_t)H * dv, dv, sb);
}

// ---------------------------------------------------------------------------
// gdn_chunk_wy_fused: build A -> approximate inverse -> W, U, on chip

template <int NB, typename F, typename TIO>
__global__ __launch_bounds__(64) void k_fused(const TIO* __restrict__ K,
                                              const TIO* __restrict__ V,
                                              const float* __restrict__ beta,
                                              const float* __restrict__ g, TIO* __restrict__ W,
                                              TIO* __restrict__ U, TIO* __restrict__ Tout, int L,
                                              int H, int dk, int dv, int N, int S) {
  constexpr int C = 16 * NB, NL = nlower(NB);
  __shared__ float sb[C], sg[C];
  const int64_t tile = blockIdx.x;
  const Chunk ch(tile, L, H, C);
  load_gates<C>(beta, g, ch, L, H, sb, sg);

  F LQ[NL], LC[NL];
  {
    f32x4 G[NL];
    gram_lower<NB, false, F>(G, K + ch.row(0, L, H, dk), (int64_t)H * dk, dk);
    gate_scale<NB, false>(G, sb, sg, -1.f);  // Lm = -A, column form
    cvt_all<NB>(LC, G);
    to_row<NB>(G, LC, 1, C - 1);
    cvt_all<NB>(LQ, G);
  }
  f32x4 Tr[NL];
  neumann_engine<NB>(LQ, LC, N, S, Tr);
  if (Tout) store_unit_row<NB>(Tout + tile * (C * C), C, Tr);

  F Tq[NL];
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
      Tq[bidx(I, J)] = Op<F>::from(x);
    }
  apply_lower<NB>(Tq, K + ch.row(0, L, H, dk), W + ch.row(0, L, H, dk), (int64_t)H * dk, dk, sb);
  apply_lower<NB>(Tq, V + ch.row(0, L, H, dv), U + ch.row(0, L, H, dv), (int64_t)H * dv, dv, sb);
}

// ---------------------------------------------------------------------------
// launchers

template <typename F, typename TK, typename TA>
static hipError_t run_build_A(const void* K, const float* beta, const float* g, void* A,
                              int64_t n, int L, int H, int dk, int C, hipStream_t st) {
  switch (C) {
#define GDN_CASE(NB)                                                                        \
  case 16 * NB:                                                                             \
    hipLaunchKernelGGL((k_build_A<NB, F, TK, TA>), dim3((unsigned)n), dim3(64), 0, st,     \
                       (const TK*)K, beta, g, (TA*)A, L, H, dk);                            \
    return hipGetLastError();
    GDN_CASE(1)
    GDN_CASE(2)
    GDN_CASE(4)
    GDN_CASE(8)
#undef GDN_CASE
  }
  return hipErrorNotSupported;
}

hipError_t launch_build_A(const void* K, const float* beta, const float* g, void* A, int B,
                          int L, int H, int dk, int C, int k_dtype, int a_dtype, hipStream_t st) {
  const int64_t n = (int64_t)B * H * (L / C);
  if (k_dtype == 0 && a_dtype == 0)
    return run_build_A<f32x4, float, float>(K, beta, g, A, n, L, H, dk, C, st);
  if (k_dtype == 0 && a_dtype == 1)
    return run_build_A<f32x4, float, __bf16>(K, beta, g, A, n, L, H, dk, C, st);
  if (k_dtype == 1 && a_dtype == 0)
    return run_build_A<bf16x4, __bf16, float>(K, beta, g, A, n, L, H, dk, C, st);
  if (k_dtype == 1 && a_dtype == 1)
    return run_build_A<bf16x4, __bf16, __bf16>(K, beta, g, A, n, L, H, dk, C, st);
  return hipErrorNotSupported;
}

template <typename F, typename TIO>
static hipError_t run_wy(const void* T, const void* K, const void* V, const float* beta,
                         void* W, void* U, int64_t n, int L, int H, int dk, int dv, int C,
                         hipStream_t st) {
  switch (C) {
#define GDN_CASE(NB)                                                                         \
  case 16 * NB:                                                                              \
    hipLaunchKernelGGL((k_wy<NB, F, TIO>), dim3((unsigned)n), dim3(64), 0, st, (const TIO*)T, \
                       (const TIO*)K, (const TIO*)V, beta, (TIO*)W, (TIO*)U, L, H, dk, dv);  \
    return hipGetLastError();
    GDN_CASE(1)
    GDN_CASE(2)
    GDN_CASE(4)
    GDN_CASE(8)
#undef GDN_CASE
  }
  return hipErrorNotSupported;
}

hipError_t launch_wy(const void* T, const void* K, const void* V, const float* beta, void* W,
                     void* U, int B, int L, int H, int dk, int dv, int C, int dtype,
                     hipStream_t st) {
  const int64_t n = (int64_t)B * H * (L / C);
  if (dtype == 0) return run_wy<f32x4, float>(T, K, V, beta, W, U, n, L, H, dk, dv, C, st);
  if (dtype == 1) return run_wy<bf16x4, __bf16>(T, K, V, beta, W, U, n, L, H, dk, dv, C, st);
  return hipErrorNotSupported;
}

template <typename F, typename TIO>
static hipError_t run_fused(const void* K, const void* V, const float* beta, const float* g,
                            void* W, void* U, void* T, int64_t n, int L, int H, int dk, int dv,
                            int C, int N, int S, hipStream_t st) {
  switch (C) {
#define GDN_CASE(NB)                                                                           \
  case 16 * NB:                                                                                \
    hipLaunchKernelGGL((k_fused<NB, F, TIO>), dim3((unsigned)n), dim3(64), 0, st,             \
                       (const TIO*)K, (const TIO*)V, beta, g, (TIO*)W, (TIO*)U, (TIO*)T, L, H, \
                       dk, dv, N, S);                                                          \
    return hipGetLastError();
    GDN_CASE(1)
    GDN_CASE(2)
    GDN_CASE(4)
#undef GDN_CASE
  }
  return hipErrorNotSupported;
}

hipError_t launch_fused(const void* K, const void* V, const float* beta, const float* g, void* W,
                        void* U, void* T, int B, int L, int H, int dk, int dv, int C, int N,
                        int S, int dtype, hipStream_t st) {
  const int64_t n = (int64_t)B * H * (L / C);
  if (dtype == 0)
    return run_fused<f32x4, float>(K, V, beta, g, W, U, T, n, L, H, dk, dv, C, N, S, st);
  if (dtype == 1)
    return run_fused<bf16x4, __bf16>(K, V, beta, g, W, U, T, n, L, H, dk, dv, C, N, S, st);
  return hipErrorNotSupported;
}

}  // namespace gdn
