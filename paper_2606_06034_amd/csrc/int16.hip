// int16.hip -- the INT16 path: per-tile quantiser and the integer
// masked-Neumann + residual inverse with 16-bit codes (Algorithm 1 with the
// INT16 activations of Section 3.5 and Appendix G of arXiv 2606.06034), one
// wave per tile; and the forward-substitution baseline on integer codes.
//
// Arithmetic: the integer reading of the INT8 path with 16-bit codes:
//   * codes q in [-32639, 32639], one exponent per tile (value q 2^e);
//   * the scale rule: q = round-half-even(v / 2^e) with e the smallest
//     integer at which no code leaves [-32639, 32639];
//   * every operator evaluated exactly from its operands' codes and its
//     result quantised once; the order, the mask and the forms as in the
//     INT8 path.
//
// gfx950 has no 16-bit integer MFMA.  32639 = 127 * 256 + 127, so every code
// splits into two int8 limbs q = 256 h + l (l in [-128, 127], h in
// [-127, 127]) and a product of codes is four int8 MFMAs over the quad
// fragments of intq.hpp (quads per limb, packed straight from the codes):
//   X Y = 2^16 Xh Yh + 2^8 (Xh Yl + Xl Yh) + Xl Yl,
// with 2^8 Xh Yh + (Xh Yl + Xl Yh) exact in int32 (|.| < 2^29) and the sum
// exact in fp64 (|X Y| < C 2^30 <= 2^36).  Products and sums are held as
// fp64 integers (exact below 2^53), codes as int32.
#include "chunk.hpp"
#include "int128.hpp"
#include "intq.hpp"
#include "int16_ops.hpp"
#include "launch.hpp"

namespace gdn {
namespace i16 {

using namespace iq;

// four int16 <-> two dwords
__device__ __forceinline__ int2 pack4_16(i32x4 x) {
  return int2{(int)((uint32_t)(x[0] & 0xffff) | ((uint32_t)x[1] << 16)),
              (int)((uint32_t)(x[2] & 0xffff) | ((uint32_t)x[3] << 16))};
}
__device__ __forceinline__ i32x4 unpack4_16(int2 w) {
  return i32x4{(int)(int16_t)(w.x & 0xffff), w.x >> 16, (int)(int16_t)(w.y & 0xffff), w.y >> 16};
}

// Tq (codes, zero above the diagonal and, in split form, on it), eT and
// optionally Tdeq = T_hat in fp32 (I + Tq 2^eT in split form, Tq 2^eT in
// plain form) for tile `tile`
template <int NB, bool PLAIN = false>
__device__ __forceinline__ void store_i16(const AccI<NB>& Tr, int eTo, int16_t* __restrict__ Tq,
                                          int32_t* __restrict__ eT, float* __restrict__ Tdeq,
                                          int64_t tile) {
  constexpr int C = 16 * NB;
  const int g = lane_g(), c = lane_c();
  int16_t* t = Tq + tile * (C * C);
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J)
      *(int2*)(t + (I * 16 + c) * C + J * 16 + 4 * g) =
          J <= I ? pack4_16(Tr.a[bidx(I, J)]) : int2{0, 0};
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

// Two waves per SIMD (amdgpu_waves_per_eu): at C = 64 the engine needs more
// than 256 registers, one wave per SIMD; held to 256 the compiler keeps
// about 120 values in scratch memory, and the second wave hides more latency
// than the scratch traffic costs (4 % less time on 32768 tiles; the one-launch
// kernel, whose K loads compete with that traffic, is faster without it).
template <int NB, bool PLAIN, int NC = -1, int SC = -1>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2)))
void k_neumann_i16(const int16_t* __restrict__ Aq,
                                                    const int32_t* __restrict__ eA,
                                                    int16_t* __restrict__ Tq,
                                                    int32_t* __restrict__ eT,
                                                    float* __restrict__ Tdeq, int Nrt, int Srt) {
  constexpr int C = 16 * NB;
  const int64_t tile = blockIdx.x;
  const int g = lane_g(), c = lane_c();
  const int16_t* a = Aq + tile * (C * C);
  // ---- Lm = -A (row form), strictly lower
  AccI<NB> Lr;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      i32x4 x = unpack4_16(*(const int2*)(a + (I * 16 + c) * C + J * 16 + 4 * g));
#pragma unroll
      for (int v = 0; v < 4; ++v) x[v] = drow(I - J, v) > 0 ? -x[v] : 0;
      Lr.a[bidx(I, J)] = x;
    }
  const int eL = __builtin_amdgcn_readfirstlane(eA[tile]);
  AccI<NB> Tr;
  int eTo;
  int_engine<I16Ops, NB, PLAIN, NC, SC>(Lr, eL, Nrt, Srt, Tr, eTo);
  store_i16<NB, PLAIN>(Tr, eTo, Tq, eT, Tdeq, tile);
}


// The whole INT16 path for one chunk in one wave: A in fp32 from K, beta, g
// (the values gdn_build_A writes), quantised in registers, then the integer
// inverse.
template <int NB, int DK, typename F, typename TK, int NC = -1, int SC = -1>
__global__ __launch_bounds__(64) void k_inverse_i16_fused(const TK* __restrict__ K,
                                                          const float* __restrict__ beta,
                                                          const float* __restrict__ g,
                                                          int16_t* __restrict__ Tq,
                                                          int32_t* __restrict__ eT,
                                                          float* __restrict__ Tdeq, int L, int H,
                                                          int Nrt, int Srt) {
  __shared__ float sb[16 * NB], sg[16 * NB];
  const Chunk ch = Chunk::by_rows(blockIdx.x, gridDim.x, L, H, 16 * NB);
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
  int_engine<I16Ops, NB, false, NC, SC>(Lr, e, Nrt, Srt, Tr, eTo);
  store_i16<NB>(Tr, eTo, Tq, eT, Tdeq, ch.tile);
}

// ---------------------------------------------------------------------------
// The INT16 width at C = 128 (k_neumann_int128, k_quantize_int128): the
// engine's limb fragments plus full 64 x 64 blocks with products as fp64
// integers.

struct FullD {
  f64x4 a[16];  // block (I, J) at 4 I + J
};

__device__ __forceinline__ void to_rowl_full(RowL<4>& X, const FullI& D) {
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int K = 0; K < 4; ++K) {
      X.h.r[I].v[K] = pack_hi(D.a[4 * I + K]);
      X.l.r[I].v[K] = pack_lo(D.a[4 * I + K]);
    }
}

// D = X Y exactly over the output block columns J0 .. J0 + JN - 1 (the
// other blocks of D are left as they are); OUTQ: row-form result
template <bool OUTQ, int J0, int JN>
__device__ __forceinline__ void mml_full(FullD& D, const RowL<4>& X, const ColL<4>& Y) {
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = J0; J < J0 + JN; ++J) {
      const i32x4 xh = X.h.r[I].v, xl = X.l.r[I].v, yh = Y.h.c[J].v, yl = Y.l.c[J].v;
      const i32x4 z = zero_i4();
      i32x4 hh, mx, ll;
      if constexpr (OUTQ) {
        hh = __builtin_amdgcn_mfma_i32_16x16x64_i8(yh, xh, z, 0, 0, 0);
        mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(yl, xh, z, 0, 0, 0);
        mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(yh, xl, mx, 0, 0, 0);
        ll = __builtin_amdgcn_mfma_i32_16x16x64_i8(yl, xl, z, 0, 0, 0);
      } else {
        hh = __builtin_amdgcn_mfma_i32_16x16x64_i8(xh, yh, z, 0, 0, 0);
        mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(xh, yl, z, 0, 0, 0);
        mx = __builtin_amdgcn_mfma_i32_16x16x64_i8(xl, yh, mx, 0, 0, 0);
        ll = __builtin_amdgcn_mfma_i32_16x16x64_i8(xl, yl, z, 0, 0, 0);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v)
        D.a[4 * I + J][v] = __builtin_fma((double)(hh[v] * 256 + mx[v]), 256.0, (double)ll[v]);
    }
}

struct I16W : I16Ops<4> {
  using Code = int16_t;
  using FProd = FullD;
  static __device__ __forceinline__ i32x4 load4(const int16_t* p) {
    return unpack4_16(*(const int2*)p);
  }
  static __device__ __forceinline__ void store4(int16_t* p, i32x4 q) { *(int2*)p = pack4_16(q); }
  static __device__ __forceinline__ int qexp(float amax) { return quant_exp(amax); }
  template <int NC, int SC>
  static __device__ __forceinline__ void engine(const AccI<4>& Lr, int eL, int N, int S,
                                                AccI<4>& Tr, int& eTo) {
    int_engine<I16Ops, 4, false, NC, SC>(Lr, eL, N, S, Tr, eTo);
  }
  static __device__ __forceinline__ void to_frow(Row& X, const FullI& D) { to_rowl_full(X, D); }
  // limb by limb through the identity (exact)
  static __device__ __forceinline__ void frow_to_col(Col& Y, const Row& X, const ColQ<4>& Ic) {
    FullI h, l;
    mmi_full<false>(h, X.h, Ic);
    mmi_full<false>(l, X.l, Ic);
    to_colq_full(Y.h, h);
    to_colq_full(Y.l, l);
  }
  template <bool OUTQ, int J0, int JN>
  static __device__ __forceinline__ void fmm(FProd& D, const Row& X, const Col& Y) {
    mml_full<OUTQ, J0, JN>(D, X, Y);
  }
  // the codes 256 h + l of block (I, K) of a row-form limb fragment
  static __device__ __forceinline__ i32x4 codes(const Row& X, int I, int K) {
    return unpack4(X.h.r[I].v[K]) * 256 + unpack4(X.l.r[I].v[K]);
  }
};

// quantiser: q = rne(x / 2^e), e the smallest integer at which every code
// lies in [-32639, 32639]
template <int C>
__global__ __launch_bounds__(64) void k_quantize_i16(const float* __restrict__ A,
                                                     int16_t* __restrict__ Aq,
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
  const float amax =
      __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(__ockl_wfred_max_f32(m))));
  const int e = quant_exp(amax);
  int16_t* q = Aq + tile * (C * C);
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    i32x4 r;
#pragma unroll
    for (int v = 0; v < 4; ++v) r[v] = (int)rintf(ldexpf(x[k][v], -e));
    *(int2*)(q + (k * 64 + l) * 4) = pack4_16(r);
  }
  if (l == 0) eA[tile] = e;
}

// ---------------------------------------------------------------------------
// The forward-substitution baseline on integer codes (Section 2.2's
// recurrence, one exponent per tile), for 16-bit and 8-bit codes: one lane
// per column j of X, rows in order.  Row i is the exact aligned sum of t
// (codes of -A at eA) and t X (products at eA + eX); the tile exponent grows
// by the smallest shift that fits the row, earlier rows rounded to it; the
// row's codes are one rounding of the sum.  Row i of A is wave-uniform
// (scalar loads).  Pairs of products of codes are exact in int32
// (|t x| < 2^30) and summed in fp64.

// code width: bits of |code|, alignment of sum terms, and qmax + 1/2 (the
// rounding threshold of the exponent growth; 16 significant bits at most,
// so the high dword of a maximum decides every comparison with it)
template <typename CODE> struct IntCodes;
template <> struct IntCodes<int16_t> {
  static constexpr int qbits = 15, align = 31;
  static constexpr double qhalf = 32639.5;
};
template <> struct IntCodes<int8_t> {
  static constexpr int qbits = 7, align = 23;
  static constexpr double qhalf = 127.5;
};

// round-half-even(y / 2^s), s >= 1, |y| < 2^15
__device__ __forceinline__ int rne_code(int y, int s) {
  if (s >= 16) return 0;  // |y| / 2^16 < 1/2
  return (y + (1 << (s - 1)) - 1 + ((y >> s) & 1)) >> s;
}

// code k of row i of a tile, read as a whole 32-bit word (wave-uniform
// addresses go through the scalar unit)
template <int C>
__device__ __forceinline__ int code_at(const int16_t* __restrict__ a, int i, int k) {
  const uint32_t w = reinterpret_cast<const uint32_t*>(a)[(i * C + k) >> 1];
  return (k & 1) ? ((int)w >> 16) : (int)(int16_t)(w & 0xffff);
}
template <int C>
__device__ __forceinline__ int code_at(const int8_t* __restrict__ a, int i, int k) {
  const uint32_t w = reinterpret_cast<const uint32_t*>(a)[(i * C + k) >> 2];
  return (int)(int8_t)(w >> (8 * (k & 3)));
}

template <int C, typename CODE>
__global__ __launch_bounds__(64) void k_fwdsub_int(const CODE* __restrict__ Aq,
                                                   const int32_t* __restrict__ eA,
                                                   CODE* __restrict__ Tq,
                                                   int32_t* __restrict__ eT,
                                                   float* __restrict__ Tdeq) {
  using Q = IntCodes<CODE>;
  constexpr int ACCB = 2 * Q::qbits + (C == 16 ? 4 : C == 32 ? 5 : 6);  // |t X| < C 2^(2 qbits)
  const int64_t tile = blockIdx.x;
  const CODE* a = Aq + tile * (C * C);
  const int j = lane_id();
  const int ea = __builtin_amdgcn_readfirstlane(eA[tile]);
  int ex = ea;
  int x[C];  // codes X_kj of this lane's column
#pragma unroll
  for (int k = 0; k < C; ++k) x[k] = 0;
  bool anyX = false;
#pragma unroll
  for (int i = 1; i < C; ++i) {
    const int tj = j < i ? -(int)a[i * C + j] : 0;
    const bool nzt = __builtin_amdgcn_ballot_w64(tj != 0) != 0;
    if (!nzt) continue;  // the row stays zero
    double p = 0.0;
#pragma unroll
    for (int k = 1; k < i; k += 2) {
      int s2 = __mul24(-code_at<C>(a, i, k), x[k]);
      if (k + 1 < i) s2 += __mul24(-code_at<C>(a, i, k + 1), x[k + 1]);
      p += (double)s2;
    }
    // aligned sum of t (first) and t X
    int es = ea + Q::qbits - Q::align;
    double acc = (double)tj * (double)(1 << (Q::align - Q::qbits));  // t 2^(ea - es)
    if (anyX) {
      const int top = ea + ex + ACCB - Q::align;
      if (top > es) {
        acc = rint(acc * ldexp(1.0, es - top));
        es = top;
      }
      const int sh = ea + ex - es;
      acc += sh >= 0 ? p * ldexp(1.0, sh) : rint(p * ldexp(1.0, sh));
    }
    // grow the tile exponent until the row fits; round the earlier rows
    const int amax_hi = wave_max(__double2hiint(fabs(acc)));
    if (amax_hi > 0) {
      int pe;
      const double m = frexp(__hiloint2double(amax_hi, 0), &pe);
      const int s = max(0, pe - Q::qbits + (m * (double)(1 << Q::qbits) >= Q::qhalf ? 1 : 0) -
                               (ex - es));
      if (s > 0) {
        int nz = 0;
#pragma unroll
        for (int k = 1; k < i; ++k) {
          x[k] = rne_code(x[k], s);
          nz |= x[k];
        }
        ex += s;
        anyX = __builtin_amdgcn_ballot_w64(nz != 0) != 0;
      }
    }
    x[i] = (int)rint(acc * ldexp(1.0, es - ex));
    anyX = anyX || __builtin_amdgcn_ballot_w64(x[i] != 0) != 0;
  }
  if (j < C) {
    CODE* t = Tq + tile * (C * C);
#pragma unroll
    for (int i = 0; i < C; ++i) t[i * C + j] = (CODE)x[i];
    if (Tdeq) {
      float* td = Tdeq + tile * (C * C);
#pragma unroll
      for (int i = 0; i < C; ++i) td[i * C + j] = i == j ? 1.f : ldexpf((float)x[i], ex);
    }
  }
  if (j == 0) eT[tile] = ex;
}

}  // namespace i16

hipError_t launch_quantize_i16(const float* A, int16_t* Aq, int32_t* eA, int64_t n, int C,
                               hipStream_t st) {
  switch (C) {
    case 16:
      hipLaunchKernelGGL((i16::k_quantize_i16<16>), dim3((unsigned)n), dim3(64), 0, st, A, Aq, eA);
      return hipGetLastError();
    case 32:
      hipLaunchKernelGGL((i16::k_quantize_i16<32>), dim3((unsigned)n), dim3(64), 0, st, A, Aq, eA);
      return hipGetLastError();
    case 64:
      hipLaunchKernelGGL((i16::k_quantize_i16<64>), dim3((unsigned)n), dim3(64), 0, st, A, Aq, eA);
      return hipGetLastError();
    case 128:
      hipLaunchKernelGGL((iq::k_quantize_int128<i16::I16W>), dim3((unsigned)n), dim3(256), 0, st,
                         A, Aq, eA);
      return hipGetLastError();
  }
  return hipErrorNotSupported;
}

namespace i16 {

// C = 16, 32: 64 / C tiles per wave (no idle lanes), the same arithmetic:
// lane l takes column l % C of tile l / C; the wave's codes are staged in
// LDS (coalesced 32-bit loads), a row of a tile is read four codes per LDS
// read, and the wave-wide maxima and "any" tests of the one-tile kernel are
// taken over the C lanes of a tile (xor-shuffles inside aligned groups).
template <int C>
__device__ __forceinline__ int group_max(int x) {
#pragma unroll
  for (int d = 1; d < C; d <<= 1) x = max(x, __shfl_xor(x, d));
  return x;
}

template <int C, typename CODE>
__global__ __launch_bounds__(64) void k_fwdsub_int_packed(const CODE* __restrict__ Aq,
                                                          const int32_t* __restrict__ eA,
                                                          CODE* __restrict__ Tq,
                                                          int32_t* __restrict__ eT,
                                                          float* __restrict__ Tdeq,
                                                          int64_t n_tiles) {
  using Q = IntCodes<CODE>;
  constexpr int P = 64 / C, PW = 4 / (int)sizeof(CODE);  // tiles per wave, codes per word
  constexpr int ACCB = 2 * Q::qbits + (C == 16 ? 4 : 5);  // |t X| < C 2^(2 qbits)
  __shared__ __attribute__((aligned(16))) int sa[P * C * C];
  const int l = threadIdx.x;
  const int64_t tile0 = (int64_t)blockIdx.x * P;
  const int64_t here = n_tiles - tile0 < P ? n_tiles - tile0 : P;
#pragma unroll
  for (int r = 0; r < (P * C * C) / (64 * PW); ++r) {
    const int w = r * 64 + l, idx = w * PW;  // word of the wave's tiles, its first code
    const uint32_t v = idx / (C * C) < here
                           ? reinterpret_cast<const uint32_t*>(Aq + tile0 * (C * C))[w]
                           : 0u;
#pragma unroll
    for (int u = 0; u < PW; ++u)
      sa[idx + u] = PW == 4 ? (int)(int8_t)(v >> (8 * u)) : (int)(int16_t)(v >> (16 * u));
  }
  __syncthreads();
  const int q = l / C, j = l % C;
  const bool live = q < here;
  const int* ar = sa + q * (C * C);
  const int ea = live ? eA[tile0 + q] : 0;
  int ex = ea;
  int x[C];
#pragma unroll
  for (int k = 0; k < C; ++k) x[k] = 0;
  bool anyX = false;
#pragma unroll
  for (int i = 1; i < C; ++i) {
    int row[C];
#pragma unroll
    for (int k0 = 0; k0 < i; k0 += 4) {
      const i32x4 r4 = *(const i32x4*)(ar + i * C + k0);
#pragma unroll
      for (int u = 0; u < 4; ++u) row[k0 + u] = r4[u];
    }
    const int tj = j < i ? -ar[i * C + j] : 0;
    double p = 0.0;
#pragma unroll
    for (int k = 1; k < i; k += 2) {
      int s2 = __mul24(-row[k], x[k]);
      if (k + 1 < i) s2 += __mul24(-row[k + 1], x[k + 1]);
      p += (double)s2;
    }
    // aligned sum of t (first) and t X (a zero row gives acc = 0, no
    // exponent growth and a zero row of codes, as the one-tile kernel's skip)
    int es = ea + Q::qbits - Q::align;
    double acc = (double)tj * (double)(1 << (Q::align - Q::qbits));
    if (anyX) {
      const int top = ea + ex + ACCB - Q::align;
      if (top > es) {
        acc = rint(acc * ldexp(1.0, es - top));
        es = top;
      }
      const int sh = ea + ex - es;
      acc += sh >= 0 ? p * ldexp(1.0, sh) : rint(p * ldexp(1.0, sh));
    }
    const int amax_hi = group_max<C>(__double2hiint(fabs(acc)));
    if (amax_hi > 0) {
      int pe;
      const double m = frexp(__hiloint2double(amax_hi, 0), &pe);
      const int sft = max(0, pe - Q::qbits + (m * (double)(1 << Q::qbits) >= Q::qhalf ? 1 : 0) -
                                 (ex - es));
      if (sft > 0) {
        int nz = 0;
#pragma unroll
        for (int k = 1; k < i; ++k) {
          x[k] = rne_code(x[k], sft);
          nz |= x[k];
        }
        ex += sft;
        anyX = group_max<C>(nz != 0 ? 1 : 0) != 0;
      }
    }
    x[i] = (int)rint(acc * ldexp(1.0, es - ex));
    anyX = anyX || group_max<C>(x[i] != 0 ? 1 : 0) != 0;
  }
  if (live) {
    CODE* t = Tq + (tile0 + q) * (C * C);
#pragma unroll
    for (int i = 0; i < C; ++i) t[i * C + j] = (CODE)x[i];
    if (Tdeq) {
      float* td = Tdeq + (tile0 + q) * (C * C);
#pragma unroll
      for (int i = 0; i < C; ++i) td[i * C + j] = i == j ? 1.f : ldexpf((float)x[i], ex);
    }
    if (j == 0) eT[tile0 + q] = ex;
  }
}

}  // namespace i16

template <typename CODE>
static hipError_t run_fwdsub_int(const CODE* Aq, const int32_t* eA, CODE* Tq, int32_t* eT,
                                 float* Tdeq, int64_t n, int C, hipStream_t st) {
  switch (C) {
    case 16:
      hipLaunchKernelGGL((i16::k_fwdsub_int_packed<16, CODE>), dim3((unsigned)((n + 3) / 4)),
                         dim3(64), 0, st, Aq, eA, Tq, eT, Tdeq, n);
      return hipGetLastError();
    case 32:
      hipLaunchKernelGGL((i16::k_fwdsub_int_packed<32, CODE>), dim3((unsigned)((n + 1) / 2)),
                         dim3(64), 0, st, Aq, eA, Tq, eT, Tdeq, n);
      return hipGetLastError();
    case 64:
      hipLaunchKernelGGL((i16::k_fwdsub_int<64, CODE>), dim3((unsigned)n), dim3(64), 0, st, Aq,
                         eA, Tq, eT, Tdeq);
      return hipGetLastError();
  }
  return hipErrorNotSupported;
}

hipError_t launch_fwdsub_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq, int32_t* eT,
                             float* Tdeq, int64_t n, int C, hipStream_t st) {
  return run_fwdsub_int<int16_t>(Aq, eA, Tq, eT, Tdeq, n, C, st);
}

hipError_t launch_fwdsub_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                            float* Tdeq, int64_t n, int C, hipStream_t st) {
  return run_fwdsub_int<int8_t>(Aq, eA, Tq, eT, Tdeq, n, C, st);
}

template <int NB, int DN, int DS>
static hipError_t run_neumann_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq, int32_t* eT,
                                  float* Tdeq, int64_t n, int N, int S, bool plain,
                                  hipStream_t st) {
  if (plain)
    hipLaunchKernelGGL((i16::k_neumann_i16<NB, true>), dim3((unsigned)n), dim3(64), 0, st, Aq,
                       eA, Tq, eT, Tdeq, N, S);
  else if (N == DN && S == DS)
    hipLaunchKernelGGL((i16::k_neumann_i16<NB, false, DN, DS>), dim3((unsigned)n), dim3(64), 0,
                       st, Aq, eA, Tq, eT, Tdeq, N, S);
  else
    hipLaunchKernelGGL((i16::k_neumann_i16<NB, false>), dim3((unsigned)n), dim3(64), 0, st, Aq,
                       eA, Tq, eT, Tdeq, N, S);
  return hipGetLastError();
}

// the default orders (3, 2), (3, 4), (3, 8) run compile-time specialisations
hipError_t launch_neumann_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq, int32_t* eT,
                              float* Tdeq, int64_t n, int C, int N, int S, bool plain,
                              hipStream_t st) {
  switch (C) {
    case 16: return run_neumann_i16<1, 3, 2>(Aq, eA, Tq, eT, Tdeq, n, N, S, plain, st);
    case 32: return run_neumann_i16<2, 3, 4>(Aq, eA, Tq, eT, Tdeq, n, N, S, plain, st);
    case 64: return run_neumann_i16<4, 3, 8>(Aq, eA, Tq, eT, Tdeq, n, N, S, plain, st);
    case 128:
      if (N == 3 && S == 8)
        hipLaunchKernelGGL((iq::k_neumann_int128<i16::I16W, 3, 8>), dim3((unsigned)n), dim3(128),
                           0, st, Aq, eA, Tq, eT, Tdeq, N, S);
      else
        hipLaunchKernelGGL((iq::k_neumann_int128<i16::I16W, -1, -1>), dim3((unsigned)n),
                           dim3(128), 0, st, Aq, eA, Tq, eT, Tdeq, N, S);
      return hipGetLastError();
  }
  return hipErrorNotSupported;
}

template <int NB, int DN, int DS, typename F, typename TK>
static hipError_t run_i16_fused(const void* K, const float* beta, const float* g, int16_t* Tq,
                                int32_t* eT, float* Tdeq, int64_t n, int L, int H, int dk, int N,
                                int S, hipStream_t st) {
#define GDN_I16F(DK, NC_, SC_)                                                               \
  hipLaunchKernelGGL((i16::k_inverse_i16_fused<NB, DK, F, TK, NC_, SC_>), dim3((unsigned)n), \
                     dim3(64), 0, st, (const TK*)K, beta, g, Tq, eT, Tdeq, L, H, N, S)
  const bool def = N == DN && S == DS;
  if (dk == 64) {
    if (def) GDN_I16F(64, DN, DS); else GDN_I16F(64, -1, -1);
  } else if (dk == 128) {
    if (def) GDN_I16F(128, DN, DS); else GDN_I16F(128, -1, -1);
  } else {
    return hipErrorNotSupported;
  }
#undef GDN_I16F
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

hipError_t launch_inverse_i16_fused(const void* K, const float* beta, const float* g,
                                    int16_t* Tq, int32_t* eT, float* Tdeq, int B, int L, int H,
                                    int dk, int C, int N, int S, int k_dtype, hipStream_t st) {
  const int64_t n = (int64_t)B * H * (L / C);
  if (C == 128)
    return run_int128_fused<i16::I16W>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, k_dtype,
                                       st);
  if (k_dtype == 1) {
    switch (C) {
      case 16: return run_i16_fused<1, 3, 2, bf16x4, __bf16>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 32: return run_i16_fused<2, 3, 4, bf16x4, __bf16>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 64: return run_i16_fused<4, 3, 8, bf16x4, __bf16>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
    }
  } else if (k_dtype == 0) {
    switch (C) {
      case 16: return run_i16_fused<1, 3, 2, f32x4, float>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 32: return run_i16_fused<2, 3, 4, f32x4, float>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
      case 64: return run_i16_fused<4, 3, 8, f32x4, float>(K, beta, g, Tq, eT, Tdeq, n, L, H, dk, N, S, st);
    }
  }
  return hipErrorNotSupported;
}

}  // namespace gdn
