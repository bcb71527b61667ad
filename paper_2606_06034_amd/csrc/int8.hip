// int8.hip -- the low-bit (INT8) path: per-tile quantiser and the integer
// masked-Neumann + residual inverse (Algorithm 1 with the integer
// activations of Section 3.5 and Appendix G of arXiv 2606.06034), one wave
// per tile.
//
// Arithmetic (the exact-integer reading the library documents):
//   * a tensor is int8 codes q in [-127, 127] with one exponent e per tile
//     (value q 2^e);
//   * the scale rule: q = round-half-even(v / 2^e) with e the smallest
//     integer at which no code leaves [-127, 127], for the quantiser of the
//     float input and for every intermediate;
//   * every operator of Algorithm 1 (MatMul, Add, the residual
//     E = I - (I + A) T0) is evaluated exactly from its operands' codes
//     (int8 x int8 products exact in int32 on v_mfma_i32_16x16x64_i8, sums
//     exact in int32 or fp64) and its result quantised once;
//   * T0 is masked once after its sum; the residual powers are
//     P_s = P_{s-1} E; T_hat = T0 T;
//   * split form: the unit diagonal of T0, T and T_hat stays out of the
//     codes; plain form (GDN_INT_PLAIN): every tensor holds its diagonal.
// Exponents and "tensor is non-zero" flags are wave-uniform (SGPRs).
//
// Operands are the int8 quad fragments of intq.hpp.
#include "chunk.hpp"
#include "int128.hpp"
#include "intq.hpp"
#include "int8_ops.hpp"
#include "launch.hpp"

namespace gdn {
namespace i8 {



// Tq (codes, zero above the diagonal and, in split form, on it), eT and
// optionally Tdeq = T_hat in fp32 (I + Tq 2^eT in split form, Tq 2^eT in
// plain form) for tile `tile`
template <int NB, bool PLAIN = false>
__device__ __forceinline__ void store_i8(const AccI<NB>& Tr, int eTo, int8_t* __restrict__ Tq,
                                         int32_t* __restrict__ eT, float* __restrict__ Tdeq,
                                         int64_t tile) {
  constexpr int C = 16 * NB;
  const int g = lane_g(), c = lane_c();
  int8_t* t = Tq + tile * (C * C);
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J)
      *(int*)(t + (I * 16 + c) * C + J * 16 + 4 * g) = J <= I ? pack4(Tr.a[bidx(I, J)]) : 0;
  if (lane_id() == 0) eT[tile] = eTo;
  if (Tdeq) {
    float* td = Tdeq + tile * (C * C);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J < NB; ++J) {
        f32x4 x = zero4();
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int d = 16 * (I - J) + c - 4 * g - v;
          if (J <= I && d >= (PLAIN ? 0 : 1)) x[v] = ldexpf((float)Tr.a[bidx(I, J)][v], eTo);
          if (!PLAIN && d == 0) x[v] = 1.f;
        }
        *(f32x4*)(td + (I * 16 + c) * C + J * 16 + 4 * g) = x;
      }
  }
}

template <int NB, bool PLAIN, int NC = -1, int SC = -1>
__global__ __launch_bounds__(64) void k_neumann_i8(const int8_t* __restrict__ Aq,
                                                   const int32_t* __restrict__ eA,
                                                   int8_t* __restrict__ Tq,
                                                   int32_t* __restrict__ eT,
                                                   float* __restrict__ Tdeq, int Nrt, int Srt) {
  constexpr int C = 16 * NB;
  const int64_t tile = blockIdx.x;
  const int g = lane_g(), c = lane_c();
  const int8_t* a = Aq + tile * (C * C);
  // ---- Lm = -A (row form), strictly lower
  AccI<NB> Lr;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      const int w = *(const int*)(a + (I * 16 + c) * C + J * 16 + 4 * g);
      i32x4 x = unpack4(w);
#pragma unroll
      for (int v = 0; v < 4; ++v) x[v] = drow(I - J, v) > 0 ? -x[v] : 0;
      Lr.a[bidx(I, J)] = x;
    }
  const int eL = __builtin_amdgcn_readfirstlane(eA[tile]);
  AccI<NB> Tr;
  int eTo;
  int_engine<I8Ops, NB, PLAIN, NC, SC>(Lr, eL, Nrt, Srt, Tr, eTo);
  store_i8<NB, PLAIN>(Tr, eTo, Tq, eT, Tdeq, tile);
}


// The whole low-bit path for one chunk in one wave: A in fp32 from K, beta,
// g (the same values gdn_build_A writes), quantised in registers by the
// quantiser's rule, then the integer inverse.
template <int NB, int DK, typename F, typename TK, int NC = -1, int SC = -1>
__global__ __launch_bounds__(64) void k_inverse_i8_fused(const TK* __restrict__ K,
                                                         const float* __restrict__ beta,
                                                         const float* __restrict__ g,
                                                         int8_t* __restrict__ Tq,
                                                         int32_t* __restrict__ eT,
                                                         float* __restrict__ Tdeq, int L, int H,
                                                         int Nrt, int Srt) {
  constexpr int C = 16 * NB;
  __shared__ float sb[C], sg[C];
  const Chunk ch = Chunk::by_rows(blockIdx.x, gridDim.x, L, H, C);
  Acc<NB> G;
  build_A_rows<NB, DK, F>(K, beta, g, ch, L, H, sb, sg, G);
  float m = 0.f;
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) m = fmaxf(m, fabsf(G.a[b][v]));
  const float amax =
      __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(__ockl_wfred_max_f32(m))));
  const int e = quant_exp(amax);
  AccI<NB> Lr;
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) Lr.a[b][v] = -(int)rintf(ldexpf(G.a[b][v], -e));
  AccI<NB> Tr;
  int eTo;
  int_engine<I8Ops, NB, false, NC, SC>(Lr, e, Nrt, Srt, Tr, eTo);
  store_i8<NB>(Tr, eTo, Tq, eT, Tdeq, ch.tile);
}

// ---------------------------------------------------------------------------
// The INT8 width at C = 128 (k_neumann_int128, k_quantize_int128): the
// engine's fragments plus full 64 x 64 blocks with exact int32 products.

struct I8W : I8Ops<4> {
  using Code = int8_t;
  using FProd = FullI;
  static __device__ __forceinline__ i32x4 load4(const int8_t* p) { return unpack4(*(const int*)p); }
  static __device__ __forceinline__ void store4(int8_t* p, i32x4 q) { *(int*)p = pack4(q); }
  static __device__ __forceinline__ int qexp(float amax) { return quant_exp(amax); }
  template <int NC, int SC>
  static __device__ __forceinline__ void engine(const AccI<4>& Lr, int eL, int N, int S,
                                                AccI<4>& Tr, int& eTo) {
    int_engine<I8Ops, 4, false, NC, SC>(Lr, eL, N, S, Tr, eTo);
  }
  static __device__ __forceinline__ void to_frow(Row& X, const FullI& D) { to_rowq_full(X, D); }
  static __device__ __forceinline__ void frow_to_col(Col& Y, const Row& X, const ColQ<4>& Ic) {
    FullI t;
    mmi_full<false>(t, X, Ic);
    to_colq_full(Y, t);
  }
  template <bool OUTQ, int J0, int JN>
  static __device__ __forceinline__ void fmm(FProd& D, const Row& X, const Col& Y) {
    mmi_full<OUTQ, J0, JN>(D, X, Y);
  }
  // the codes of block (I, K) of a row-form fragment
  static __device__ __forceinline__ i32x4 codes(const Row& X, int I, int K) {
    return unpack4(X.r[I].v[K]);
  }
};

// ---------------------------------------------------------------------------
// quantiser: q = rne(x / 2^e), e the smallest integer at which every code
// lies in [-127, 127]

template <int C>
__global__ __launch_bounds__(64) void k_quantize_i8(const float* __restrict__ A,
                                                    int8_t* __restrict__ Aq,
                                                    int32_t* __restrict__ eA) {
  constexpr int PER = C * C / 64 / 4;  // float4 per lane
  const int64_t tile = blockIdx.x;
  const float* a = A + tile * (C * C);
  const int l = lane_id();
  f32x4 x[PER];
  float m = 0.f;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int idx = (k * 64 + l) * 4;
    x[k] = *(const f32x4*)(a + idx);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = (idx + v) / C, j = (idx + v) % C;
      if (i <= j) x[k][v] = 0.f;
      m = fmaxf(m, fabsf(x[k][v]));
    }
  }
  const float amax = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(__ockl_wfred_max_f32(m))));
  const int e = quant_exp(amax);
  int8_t* q = Aq + tile * (C * C);
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    i32x4 r;
#pragma unroll
    for (int v = 0; v < 4; ++v) r[v] = (int)rintf(ldexpf(x[k][v], -e));
    *(int*)(q + (k * 64 + l) * 4) = pack4(r);
  }
  if (l == 0) eA[tile] = e;
}

}  // namespace i8

hipError_t launch_quantize_i8(const float* A, int8_t* Aq, int32_t* eA, int64_t n, int C,
                              hipStream_t st) {
  switch (C) {
    case 16:
      hipLaunchKernelGGL((i8::k_quantize_i8<16>), dim3((unsigned)n), dim3(64), 0, st, A, Aq, eA);
      return hipGetLastError();
    case 32:
      hipLaunchKernelGGL((i8::k_quantize_i8<32>), dim3((unsigned)n), dim3(64), 0, st, A, Aq, eA);
      return hipGetLastError();
    case 64:
      hipLaunchKernelGGL((i8::k_quantize_i8<64>), dim3((unsigned)n), dim3(64), 0, st, A, Aq, eA);
      return hipGetLastError();
    case 128:
      hipLaunchKernelGGL((iq::k_quantize_int128<i8::I8W>), dim3((unsigned)n), dim3(256), 0, st, A,
                         Aq, eA);
      return hipGetLastError();
  }
  return hipErrorNotSupported;
}

template <int NB, int DN, int DS>
static hipError_t run_neumann_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                                 float* Tdeq, int64_t n, int N, int S, bool plain,
                                 hipStream_t st) {
  if (plain)
    hipLaunchKernelGGL((i8::k_neumann_i8<NB, true>), dim3((unsigned)n), dim3(64), 0, st, Aq, eA,
                       Tq, eT, Tdeq, N, S);
  else if (N == DN && S == DS)
    hipLaunchKernelGGL((i8::k_neumann_i8<NB, false, DN, DS>), dim3((unsigned)n), dim3(64), 0, st,
                       Aq, eA, Tq, eT, Tdeq, N, S);
  else
    hipLaunchKernelGGL((i8::k_neumann_i8<NB, false>), dim3((unsigned)n), dim3(64), 0, st, Aq, eA,
                       Tq, eT, Tdeq, N, S);
  return hipGetLastError();
}

// the default orders (3, 2), (3, 4), (3, 8) of the split form run
// compile-time specialisations; plain form only at C <= 64
hipError_t launch_neumann_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                             float* Tdeq, int64_t n, int C, int N, int S, bool plain,
                             hipStream_t st) {
  switch (C) {
    case 16: return run_neumann_i8<1, 3, 2>(Aq, eA, Tq, eT, Tdeq, n, N, S, plain, st);
    case 32: return run_neumann_i8<2, 3, 4>(Aq, eA, Tq, eT, Tdeq, n, N, S, plain, st);
    case 64: return run_neumann_i8<4, 3, 8>(Aq, eA, Tq, eT, Tdeq, n, N, S, plain, st);
    case 128:
      if (N == 3 && S == 8)
        hipLaunchKernelGGL((iq::k_neumann_int128<i8::I8W, 3, 8>), dim3((unsigned)n), dim3(128), 0,
                           st, Aq, eA, Tq, eT, Tdeq, N, S);
      else
        hipLaunchKernelGGL((iq::k_neumann_int128<i8::I8W, -1, -1>), dim3((unsigned)n), dim3(128),
                           0, st, Aq, eA, Tq, eT, Tdeq, N, S);
      return hipGetLastError();
  }
  return hipErrorNotSupported;
}

template <int NB, int DN, int DS, typename F, typename TK>
static hipError_t run_i8_fused(const void* K, const float* beta, const float* g, int8_t* Tq,
                               int32_t* eT, float* Tdeq, int64_t n, int L, int H, int dk, int N,
                               int S, hipStream_t st) {
#define GDN_I8F(DK, NC_, SC_)                                                                \
  hipLaunchKernelGGL((i8::k_inverse_i8_fused<NB, DK, F, TK, NC_, SC_>), dim3((unsigned)n),   \
                     dim3(64), 0, st, (const TK*)K, beta, g, Tq, eT, Tdeq, L, H, N, S)
  const bool def = N == DN && S == DS;
  if (dk == 64) {
    if (def) GDN_I8F(64, DN, DS); else GDN_I8F(64, -1, -1);
  } else if (dk == 128) {
    if (def) GDN_I8F(128, DN, DS); else GDN_I8F(128, -1, -1);
  } else {
    return hipErrorNotSupported;
  }
#undef GDN_I8F
  return hipGetLastError();
}

// C = 128 in one launch (k_inverse_int128_fused), two waves per tile
template <typename W>
static hipError_t run_int128_fused(const void* K, const float* beta, const float* g,
                                   typename W::Code* Tq, int32_t* eT, float* Tdeq, int64_t n,
                                   int L, int H, int dk, int N, int S, int k_dtype,
                                   hipStream_t st) {
#define GDN_I128F(DK, F, TK, NC_, SC_)                                                         \
  hipLaunchKernelGGL((iq::k_inverse_int128_fused<W, DK, F, TK, NC_, SC_>), dim3((unsigned)n), \
                     dim3(128), 0, st, (const TK*)K, beta, g, Tq, eT, Tdeq, L, H, N, S)
#define GDN_I128F_ORD(DK, F, TK)                       \
  if (N == 3 && S == 8) GDN_I128F(DK, F, TK, 3, 8);   \
  else GDN_I128F(DK, F, TK, -1, -1)
  if (k_dtype == 1) {
    if (dk == 64) { GDN_I128F_ORD(64, bf16x4, __bf16); }
    else if (dk == 128) { GDN_I128F_ORD(128, bf16x4, __bf16); }
    else return hipErrorNotSupported;
  } else if (k_dtype == 0) {
    if (dk == 64) { GDN_I128F_ORD(64, f32x4, float); }
    else if (dk == 128) { GDN_I128F_ORD(128, f32x4, float); }
    else return hipErrorNotSupported;
  } else {
    return hipErrorNotSupported;
  }
#undef GDN_I128F_ORD
#undef GDN_I128F
  return hipGetLastError();
}

hipError_t launch_inverse_i8_fused(const void* K, const float* beta, const float* g, int8_t* Tq,
                                   int32_t* eT, float* Tdeq, int B, int L, int H, int dk, int C,
                                   int N, int S, int k_dtype, hipStream_t st) {
  const int64_t n = (int64_t)B * H * (L / C);
  if (C == 128)
    return run_int128_fused<i8::I8W>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, k_dtype, st);
  if (k_dtype == 1) {
    switch (C) {
      case 16: return run_i8_fused<1, 3, 2, bf16x4, __bf16>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 32: return run_i8_fused<2, 3, 4, bf16x4, __bf16>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 64: return run_i8_fused<4, 3, 8, bf16x4, __bf16>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
    }
  } else if (k_dtype == 0) {
    switch (C) {
      case 16: return run_i8_fused<1, 3, 2, f32x4, float>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 32: return run_i8_fused<2, 3, 4, f32x4, float>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 64: return run_i8_fused<4, 3, 8, f32x4, float>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
    }
  }
  return hipErrorNotSupported;
}

}  // namespace gdn
