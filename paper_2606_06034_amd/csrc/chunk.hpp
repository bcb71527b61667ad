// chunk.hpp -- per-chunk input handling shared by the kernels that start
// from K, beta, g in the [B, L, H, d] layouts: the work-item to chunk map,
// gate staging, 16-byte row loads and the Gram product with the gates
// (A_ij = beta_i (k_i . k_j) exp(g_i - g_j) for i > j, Section 2.1).
#pragma once

#include "tile16.hpp"

namespace gdn {

// Chunk bookkeeping.  Work item x walks the tiles heads-fastest,
// x = (b * (L / C) + chunk) * H + h, so waves running side by side read the
// neighbouring heads of the same tokens: together they cover whole
// H * d-wide token rows of [B, L, H, d] instead of one 256-byte run per row
// and DRAM page (+10 % bandwidth for this access pattern on MI355X).
// `tile` is the position in the [B, H, L/C, C, C] tile layout.
struct Chunk {
  int b, h, t0;
  int m;  // rows holding tokens: C, or fewer in the last chunk of a packed sequence
  int64_t tile;
  __device__ Chunk() {}
  // x < 2^31 (the tile count is bounded so): 32-bit unsigned division.
  // Workgroups are dealt round-robin to the 8 XCDs (x % 8).  When H is a
  // multiple of 8, XCD k takes the heads k H/8 .. (k+1) H/8 - 1 of every
  // token row (heads fastest inside its group), so each XCD streams its own
  // contiguous H/8 * d-wide column band of [B, L, H, d]: a copy with this
  // addressing runs 6 % faster on MI355X than with the heads dealt across
  // the XCDs.  A bijection of the work items; tiles are unchanged.
  __device__ Chunk(uint32_t x, int L, int H, int C, bool bands = true) {
    const uint32_t nc = (uint32_t)(L / C);
    if (bands && (H & 7) == 0) {
      const uint32_t hg = (uint32_t)H >> 3, slot = x >> 3;
      const uint32_t row = slot / hg;
      x = row * (uint32_t)H + (x & 7u) * hg + (slot - row * hg);
    }
    const uint32_t bc = x / (uint32_t)H;
    h = (int)(x - bc * (uint32_t)H);
    b = (int)(bc / nc);
    const int chunk = (int)(bc - (uint32_t)b * nc);
    t0 = chunk * C;
    m = C;
    tile = ((int64_t)b * H + h) * nc + chunk;
  }
  // The work-item map of the compute-bound integer kernels, n = B H (L / C)
  // work items: XCD k (x % 8) takes every H-th group of work items whole, so
  // all heads of chunk rows k, k + 8, k + 16, ... run on one XCD and a gate
  // cache line (the H heads of one token) is fetched once, not once per
  // XCD; with the heads of a row dealt across the XCDs, gate reads are 8
  // times the algorithmic bytes.  A partial last group of fewer than 8 rows
  // keeps the plain order.  A bijection of the work items; tiles unchanged.
  static __device__ Chunk by_rows(uint32_t x, uint32_t n, int L, int H, int C) {
    const uint32_t hh = (uint32_t)H, R8 = (n / hh) & ~7u;
    if (x < R8 * hh) {
      const uint32_t s = x >> 3, grp = s / hh;
      x = (8u * grp + (x & 7u)) * hh + (s - grp * hh);
    }
    return Chunk(x, L, H, C, false);
  }
  // Work item of wave w of workgroup wg when workgroups hold G waves (G
  // divides H / 8): the waves of one workgroup take consecutive slots of the
  // XCD wg % 8, i.e. G neighbouring heads of one chunk row of that XCD's
  // head band (the map of the constructor above), and the workgroup stays on
  // the XCD its tiles belong to.
  static __device__ uint32_t grouped(uint32_t wg, int w, int G) {
    return ((((wg >> 3) * (uint32_t)G + (uint32_t)w)) << 3) | (wg & 7u);
  }
  // Packed sequences (B = 1, T tokens): sequence s holds tokens
  // cu[s] .. cu[s + 1] - 1 and chunks off[s] .. off[s + 1] - 1, each chunk
  // starting at a multiple of C from the sequence start.  Work item
  // x = chunk * H + h; tile = h * nchunks + chunk.  Inconsistent tables give
  // m = 0 (nothing to do), never an access outside the T tokens.
  static __device__ Chunk packed(uint32_t x, int H, int C, int T, const int* __restrict__ cu,
                                 const int* __restrict__ off, int nseq, int nchunks) {
    Chunk ch;
    const int chunk = (int)(x / (uint32_t)H);
    ch.h = (int)(x - (uint32_t)chunk * (uint32_t)H);
    ch.b = 0;
    ch.tile = (int64_t)ch.h * nchunks + chunk;
    // the last s with off[s] <= chunk (empty sequences repeat an offset)
    int lo = 0, hi = nseq;  // off[lo] <= chunk is assumed, off[hi] = nchunks > chunk
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (off[mid] <= chunk) lo = mid; else hi = mid;
    }
    const int64_t t0 = (int64_t)cu[lo] + (int64_t)(chunk - off[lo]) * C;
    const int64_t end = min((int64_t)cu[lo + 1], (int64_t)T);
    ch.t0 = (t0 >= 0 && t0 < T) ? (int)t0 : 0;
    ch.m = (t0 >= 0 && t0 < T) ? (int)max((int64_t)0, min((int64_t)C, end - t0)) : 0;
    return ch;
  }
  // element offset of (token t0 + r, head h, feature 0) in [B, L, H, d]
  __device__ int64_t row(int r, int L, int H, int d) const {
    return (((int64_t)b * L + t0 + r) * H + h) * d;
  }
};

// Packed sequences: cu (nseq + 1 token offsets) and off (nseq + 1 chunk
// offsets) device tables; nullptr for the fixed-length layout.
struct Packed {
  const int* cu = nullptr;
  const int* off = nullptr;
  int nseq = 0, nchunks = 0;
};

// beta and g of the chunk into LDS (one wave; C <= 128).  Rows r >= m (past
// the end of a packed sequence) get beta = 0, which makes them write nothing
// (A's rows vanish, T is the identity there), and the last row's g.
// Orders LDS writes before the reads that follow: within one wave (WAVE:
// the data is this wave's own) or across the workgroup.
template <bool WAVE>
__device__ __forceinline__ void lds_sync() {
  if constexpr (WAVE) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();
  }
}

// In two steps, so that a kernel can issue its K loads between them: the
// LDS writes wait for the gate loads, and the barrier must not hold back
// the next loads behind a second memory latency.
template <int C> struct GateRows {
  static constexpr int R = (C + 63) / 64;  // rows per lane
  float b[R], g[R];
};
template <int C>
__device__ __forceinline__ GateRows<C> fetch_gates(const float* __restrict__ beta,
                                                   const float* __restrict__ g, const Chunk& ch,
                                                   int L, int H, int m = C) {
  GateRows<C> gr;
#pragma unroll
  for (int k = 0; k < GateRows<C>::R; ++k) {
    const int r = lane_id() + 64 * k;
    const int rr = r < C ? (r < m ? r : m - 1) : 0;
    const int64_t o = ((int64_t)ch.b * L + ch.t0 + rr) * H + ch.h;
    gr.b[k] = (r < C && r < m && beta) ? beta[o] : 0.f;
    gr.g[k] = (r < C && g) ? g[o] : 0.f;
  }
  return gr;
}
// WAVE: the gates are read by this wave only (its own LDS arrays in a
// workgroup of several waves), so a wave barrier orders its lanes' LDS
// writes before their reads instead of a workgroup barrier.
template <int C, bool WAVE = false>
__device__ __forceinline__ void stash_gates(const GateRows<C>& gr, float* sb, float* sg) {
#pragma unroll
  for (int k = 0; k < GateRows<C>::R; ++k) {
    const int r = lane_id() + 64 * k;
    if (r < C) {
      if (sb) sb[r] = gr.b[k];
      if (sg) sg[r] = gr.g[k];
    }
  }
  lds_sync<WAVE>();
}
template <int C>
__device__ __forceinline__ void load_gates(const float* __restrict__ beta,
                                           const float* __restrict__ g, const Chunk& ch, int L,
                                           int H, float* sb, float* sg, int m = C) {
  stash_gates<C>(fetch_gates<C>(beta, g, ch, L, H, m), sb, sg);
}

// Lower blocks of the chunk Gram matrix K K^T (fp32 accumulation), in the
// form OUTQ selects, from the row pairs of K (load_rows): both factors are
// rows of K and any feature order serves as the contraction order.
template <int NB, int DK, bool OUTQ, typename F>
__device__ __forceinline__ void gram_lower(Acc<NB>& G, const Pair<F> (&kp)[NB][DK / 32]) {
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J) {
      f32x4 acc = zero4();
#pragma unroll
      for (int q = 0; q < DK / 32; ++q) acc = Pair<F>::template mma<OUTQ>(kp[I][q], kp[J][q], acc);
      G.a[bidx(I, J)] = acc;
    }
}

// A (times `sign`) from the Gram blocks, in place; ROWFORM selects the
// element coordinates of the blocks' form.
template <int NB, bool ROWFORM>
__device__ __forceinline__ void gate_scale(Acc<NB>& G, const float* sb, const float* sg,
                                           float sign, Lane ln = lane_here()) {
  const int g = ln.g(), c = ln.c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = ROWFORM ? I * 16 + c : I * 16 + 4 * g + v;
        const int j = ROWFORM ? J * 16 + 4 * g + v : J * 16 + c;
        const float x = G.a[bidx(I, J)][v];
        G.a[bidx(I, J)][v] = (i > j) ? sign * sb[i] * x * __expf(sg[i] - sg[j]) : 0.f;
      }
}

// 16-byte loads of a chunk of X [token][feature] (row stride ld): lane (g, c)
// gets 8 consecutive features 32q + 8g .. 32q + 8g + 7 of token 16I + c, as
// one row-form pair over two 16-feature halves.  Within chunk q the half h
// holds features 32q + 8 (j / 4) + 4h + (j % 4) in block column j, so the
// same permutation maps MFMA columns back to memory on store.
template <typename F, typename TIO>
__device__ __forceinline__ Pair<F> load_row8(const TIO* __restrict__ p);
template <>
__device__ __forceinline__ Pair<bf16x4> load_row8<bf16x4, __bf16>(const __bf16* __restrict__ p) {
  return Pair<bf16x4>{*(const bf16x8*)p};
}
template <>
__device__ __forceinline__ Pair<f32x4> load_row8<f32x4, float>(const float* __restrict__ p) {
  return Pair<f32x4>{*(const f32x4*)p, *(const f32x4*)(p + 4)};
}
__device__ __forceinline__ void store_row8(__bf16* p, f32x4 lo, f32x4 hi) {
  const bf16x4 a = __builtin_convertvector(lo, bf16x4), b = __builtin_convertvector(hi, bf16x4);
  *(bf16x8*)p = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
__device__ __forceinline__ void store_row8(float* p, f32x4 lo, f32x4 hi) {
  *(f32x4*)p = lo;
  *(f32x4*)(p + 4) = hi;
}

// Rows r >= m (past the end of a packed sequence) are read from row m - 1
// and set to 0.
template <int NB, int D, typename F, typename TIO>
__device__ __forceinline__ void load_rows(Pair<F> (&xp)[NB][D / 32], const TIO* __restrict__ xb,
                                          int64_t ld, Lane ln = lane_here(), int m = 16 * NB) {
  const int g = ln.g(), c = ln.c();
#pragma unroll
  for (int I = 0; I < NB; ++I) {
    const int r = I * 16 + c, rr = r < m ? r : m - 1;
#pragma unroll
    for (int q = 0; q < D / 32; ++q) {
      xp[I][q] = load_row8<F>(xb + rr * ld + 32 * q + 8 * g);
      if (r >= m) xp[I][q] = Pair<F>::zero();
    }
  }
}

// The strictly lower A of one chunk in fp32, row-form blocks (zero on and
// above the diagonal): Gram product of the chunk's K rows in compute type F,
// then the gates.  Every kernel that forms A from K goes through here, so
// they all produce the same fp32 values.  sb, sg: LDS arrays of C floats.
template <int NB, int DK, typename F, typename TK>
__device__ __forceinline__ void build_A_rows(const TK* __restrict__ K,
                                             const float* __restrict__ beta,
                                             const float* __restrict__ g, const Chunk& ch,
                                             int L, int H, float* sb, float* sg, Acc<NB>& G) {
  const GateRows<16 * NB> gr = fetch_gates<16 * NB>(beta, g, ch, L, H);
  {
    Pair<F> kp[NB][DK / 32];
    load_rows<NB, DK>(kp, K + ch.row(0, L, H, DK), (int64_t)H * DK);
    stash_gates<16 * NB>(gr, sb, sg);
    gram_lower<NB, DK, true>(G, kp);
  }
  gate_scale<NB, true>(G, sb, sg, 1.f);
}

}  // namespace gdn
