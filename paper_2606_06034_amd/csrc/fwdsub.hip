// fwdsub.hip -- exact (I + A)^-1 by forward substitution, the row-serial
// baseline of Section 2.2 (Eq. forward_sub) of arXiv 2606.06034.
//
// One lane per column j of the inverse X, so the C - 1 dependent row steps
// run in lock-step across the wave:
//     x_ij = -sum_{t < i} a_it x_tj   (i > j),   x_jj = 1,   x_ij = 0 (i < j).
// Row i of A is wave-uniform: it is read with scalar loads and broadcast to
// every lane as an SGPR operand, so each term is one fp32 FMA per lane.  The
// column lives in VGPRs (fully unrolled, C registers per lane).  Four
// partial sums shorten each row's dependency chain.  C = 128 uses two waves
// (columns 0..63 and 64..127); the second starts at row 64, where its
// columns first become non-zero.  Computed in fp32 whatever the storage type.
#include "launch.hpp"

namespace gdn {

// a[i * C + k] of a tile, read as whole 32-bit words so that a wave-uniform
// address goes through the scalar unit (bf16 pairs share one word).
template <int C>
__device__ __forceinline__ float ld1(const float* __restrict__ a, int i, int k) {
  return a[i * C + k];
}
template <int C>
__device__ __forceinline__ float ld1(const __bf16* __restrict__ a, int i, int k) {
  const uint32_t w = reinterpret_cast<const uint32_t*>(a)[(i * C + k) >> 1];
  return __uint_as_float((k & 1) ? (w & 0xffff0000u) : (w << 16));
}
__device__ __forceinline__ void st1(float* p, float x) { *p = x; }
__device__ __forceinline__ void st1(__bf16* p, float x) { *p = (__bf16)x; }

template <int C, int R0, typename TIO>
__device__ __forceinline__ void fwdsub_rows(const TIO* __restrict__ a, TIO* __restrict__ t, int j) {
  float x[C];
#pragma unroll
  for (int i = 0; i < R0; ++i) x[i] = 0.f;
#pragma unroll
  for (int i = R0; i < C; ++i) {
    float s[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = R0; k < i; ++k) s[k & 3] = fmaf(ld1<C>(a, i, k), x[k], s[k & 3]);
    const float acc = (s[0] + s[1]) + (s[2] + s[3]);
    x[i] = (i > j) ? -acc : (i == j ? 1.f : 0.f);
  }
  if (j < C) {
#pragma unroll
    for (int i = 0; i < C; ++i) st1(t + i * C + j, x[i]);
  }
}

template <int C, typename TIO>
__global__ __launch_bounds__(C < 64 ? 64 : C) void k_fwdsub(const TIO* __restrict__ A,
                                                             TIO* __restrict__ T) {
  const int64_t tile = blockIdx.x;
  const TIO* a = A + tile * (C * C);
  TIO* t = T + tile * (C * C);
  const int j = threadIdx.x;
  if constexpr (C == 128) {
    if (j >= 64)
      fwdsub_rows<C, 64>(a, t, j);
    else
      fwdsub_rows<C, 0>(a, t, j);
  } else {
    fwdsub_rows<C, 0>(a, t, j);
  }
}

template <int C, typename TIO>
static hipError_t run_fwdsub(const void* A, void* T, int64_t n, hipStream_t st) {
  hipLaunchKernelGGL((k_fwdsub<C, TIO>), dim3((unsigned)n), dim3(C < 64 ? 64 : C), 0, st,
                     (const TIO*)A, (TIO*)T);
  return hipGetLastError();
}

template <typename TIO>
static hipError_t run_fwdsub_c(const void* A, void* T, int64_t n, int C, hipStream_t st) {
  switch (C) {
    case 16: return run_fwdsub<16, TIO>(A, T, n, st);
    case 32: return run_fwdsub<32, TIO>(A, T, n, st);
    case 64: return run_fwdsub<64, TIO>(A, T, n, st);
    case 128: return run_fwdsub<128, TIO>(A, T, n, st);
  }
  return hipErrorNotSupported;
}

hipError_t launch_fwdsub(const void* A, void* T, int64_t n, int C, int dtype, hipStream_t st) {
  if (dtype == 0) return run_fwdsub_c<float>(A, T, n, C, st);
  if (dtype == 1) return run_fwdsub_c<__bf16>(A, T, n, C, st);
  return hipErrorNotSupported;
}

}  // namespace gdn
