// fwdsub.hip -- exact (I + A)^-1 by forward substitution, the row-serial
// baseline of Section 2.2 (Eq. forward_sub) of arXiv 2606.06034.
//
// One lane per column j of the inverse X, so the C - 1 dependent row steps
// run in lock-step across the wave:
//     x_ij = -sum_{t < i} a_it x_tj   (i > j),   x_jj = 1,   x_ij = 0 (i < j).
// C = 64: row i of A is wave-uniform: it is read with scalar loads and
// broadcast to every lane as an SGPR operand, so each term is one fp32 FMA
// per lane.  The column lives in VGPRs (fully unrolled, C registers per
// lane).  Four partial sums shorten each row's dependency chain.  C = 128
// uses two waves (columns 0..63 and 64..127); the second starts at row 64,
// where its columns first become non-zero.  C = 16, 32: 64 / C tiles per
// wave, so that no lane idles: the wave's tiles are staged in LDS (fp32,
// coalesced 16-byte loads) and lane l takes column l % C of tile l / C,
// reading four entries of its tile's row i per LDS read.  Computed in fp32
// whatever the storage type.
#include "launch.hpp"
#include "tile16.hpp"

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

// 16 bytes of a tile as fp32
__device__ __forceinline__ void ld_vec(const float* p, float* o) {
  const f32x4 v = *(const f32x4*)p;
#pragma unroll
  for (int u = 0; u < 4; ++u) o[u] = v[u];
}
__device__ __forceinline__ void ld_vec(const __bf16* p, float* o) {
  const bf16x8 v = *(const bf16x8*)p;
#pragma unroll
  for (int u = 0; u < 8; ++u) o[u] = (float)v[u];
}

// C = 16, 32: P = 64 / C tiles per wave (the last wave of a launch may hold
// fewer; its missing tiles read as zero and are not written)
template <int C, typename TIO>
__global__ __launch_bounds__(64) void k_fwdsub_packed(const TIO* __restrict__ A,
                                                      TIO* __restrict__ T, int64_t n_tiles) {
  constexpr int P = 64 / C, E = 16 / sizeof(TIO);  // tiles per wave, elements per 16 bytes
  __shared__ __attribute__((aligned(16))) float sa[P * C * C];
  const int l = threadIdx.x;
  const int64_t tile0 = (int64_t)blockIdx.x * P;
  const int64_t here = n_tiles - tile0 < P ? n_tiles - tile0 : P;
  // stage the wave's tiles: 64 C elements, E per lane and step, coalesced
#pragma unroll
  for (int r = 0; r < (P * C * C) / (64 * E); ++r) {
    const int idx = (r * 64 + l) * E;  // element of the wave's tiles
    float v[E];
    if (idx / (C * C) < here) {
      ld_vec(A + tile0 * (C * C) + idx, v);
    } else {
#pragma unroll
      for (int u = 0; u < E; ++u) v[u] = 0.f;
    }
#pragma unroll
    for (int u = 0; u < E; ++u) sa[idx + u] = v[u];
  }
  __syncthreads();
  const int q = l / C, j = l % C;
  const float* ar = sa + q * (C * C);
  float x[C];
#pragma unroll
  for (int i = 0; i < C; ++i) {
    float s4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k0 = 0; k0 < i; k0 += 4) {
      const f32x4 a4 = *(const f32x4*)(ar + i * C + k0);
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (k0 + u < i) s4[u] = fmaf(a4[u], x[k0 + u], s4[u]);
    }
    const float acc = (s4[0] + s4[1]) + (s4[2] + s4[3]);
    x[i] = (i > j) ? -acc : (i == j ? 1.f : 0.f);
  }
  if (q < here) {
    TIO* t = T + (tile0 + q) * (C * C);
#pragma unroll
    for (int i = 0; i < C; ++i) st1(t + i * C + j, x[i]);
  }
}

template <int C, typename TIO>
static hipError_t run_fwdsub(const void* A, void* T, int64_t n, hipStream_t st) {
  if constexpr (C < 64) {
    constexpr int P = 64 / C;
    hipLaunchKernelGGL((k_fwdsub_packed<C, TIO>), dim3((unsigned)((n + P - 1) / P)), dim3(64), 0,
                       st, (const TIO*)A, (TIO*)T, n);
  } else {
    hipLaunchKernelGGL((k_fwdsub<C, TIO>), dim3((unsigned)n), dim3(C), 0, st, (const TIO*)A,
                       (TIO*)T);
  }
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
