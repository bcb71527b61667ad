// pipeline.hip -- building A, applying the inverse to K and V (WY form), and
// the fused chunk pipeline.  One wave per (batch, head, chunk) tile.
//
//   A_ij = beta_i (k_i . k_j) exp(g_i - g_j) for i > j       (Section 2.1)
//   W = T diag(beta) K,  U = T diag(beta) V
#include "launch.hpp"
#include "wy.hpp"

namespace gdn {

// ---------------------------------------------------------------------------
// gdn_build_A

template <int NB, int DK, typename F, typename TK, typename TA>
__global__ __launch_bounds__(64) void k_build_A(const TK* __restrict__ K,
                                                const float* __restrict__ beta,
                                                const float* __restrict__ g,
                                                TA* __restrict__ A, int L, int H) {
  constexpr int C = 16 * NB;
  __shared__ float sb[C], sg[C];
  const Chunk ch(blockIdx.x, L, H, C);
  const int64_t tile = ch.tile;
  Acc<NB> G;
  build_A_rows<NB, DK, F>(K, beta, g, ch, L, H, sb, sg, G);
  TA* a = A + tile * (C * C);
  const int gg = lane_g(), c = lane_c();
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J < NB; ++J)
      store4(a + (I * 16 + c) * C + J * 16 + 4 * gg, J <= I ? G.a[bidx(I, J)] : zero4());
}

// ---------------------------------------------------------------------------
// gdn_wy_apply

template <int NB, int DK, int DV, typename F, typename TIO>
__global__ __launch_bounds__(64) void k_wy(const TIO* __restrict__ T, const TIO* __restrict__ K,
                                           const TIO* __restrict__ V,
                                           const float* __restrict__ beta, TIO* __restrict__ W,
                                           TIO* __restrict__ U, int L, int H) {
  constexpr int C = 16 * NB;
  __shared__ float sb[C];
  const Chunk ch(blockIdx.x, L, H, C);
  const int64_t tile = ch.tile;
  load_gates<C>(beta, beta, ch, L, H, sb, nullptr);
  const TIO* t = T + tile * (C * C);
  const int g = lane_g(), c = lane_c();
  Acc<NB> Tq;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
      Tq.a[bidx(I, J)] =
          band_block<false>(load4(t + (I * 16 + c) * C + J * 16 + 4 * g), I - J, 0, C);
  RowP<NB, F> TR;
  scale_cols(TR, Tq, sb);
  {
    Pair<F> kp[NB][DK / 32];
    load_rows<NB, DK>(kp, K + ch.row(0, L, H, DK), (int64_t)H * DK);
    apply_lower<NB, DK>(TR, RegRows<NB, DK, F>{kp}, W + ch.row(0, L, H, DK), (int64_t)H * DK);
  }
  {
    Pair<F> vp[NB][DV / 32];
    load_rows<NB, DV>(vp, V + ch.row(0, L, H, DV), (int64_t)H * DV);
    apply_lower<NB, DV>(TR, RegRows<NB, DV, F>{vp}, U + ch.row(0, L, H, DV), (int64_t)H * DV);
  }
}

// ---------------------------------------------------------------------------
// gdn_chunk_wy_fused: build A -> approximate inverse -> W, U, on chip

// One tile per wave.  PREF (bf16 only): V is copied into LDS by DMA right
// after the Gram product and arrives while the inverse is computed.
// VARLEN: packed sequences (B = 1, L = T tokens, chunk tables cu / off):
// the last chunk of a sequence may hold m < C tokens; its rows past m are
// neither read nor written (T is the identity there).
template <int NB, int DK, int DV, typename F, bool SMALLN, int NC, int SC, typename TIO,
          bool PREF = false, bool EXACT = false, bool VARLEN = false, int WPG = 1>
__global__ __launch_bounds__(64 * WPG) void k_fused(const TIO* __restrict__ K,
                                              const TIO* __restrict__ V,
                                              const float* __restrict__ beta,
                                              const float* __restrict__ g, TIO* __restrict__ W,
                                              TIO* __restrict__ U, TIO* __restrict__ Tout, int L,
                                              int H, int N, int S, const int* __restrict__ cu,
                                              const int* __restrict__ off, int nseq,
                                              int nchunks) {
  constexpr int C = 16 * NB;
  static_assert(!PREF || sizeof(TIO) == 2, "V prefetch is for bf16 IO");
  // WPG > 1: the workgroup's waves take neighbouring heads of one chunk row
  // (Chunk::grouped; packed sequences: G consecutive work items chunk H + h),
  // each with its own LDS arrays
  __shared__ float sb_[WPG][C], sg_[WPG][C];
  __shared__ __attribute__((aligned(16))) __bf16 sv_[WPG][PREF ? NB * (DV / 32) * 512 : 8];
  const int wv = WPG > 1 ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) : 0;
  float* sb = sb_[wv];
  float* sg = sg_[wv];
  __bf16* sv = sv_[wv];
  Chunk ch;
  if constexpr (VARLEN)
    ch = Chunk::packed(blockIdx.x * WPG + wv, H, C, L, cu, off, nseq, nchunks);
  else
    ch = Chunk(WPG > 1 ? Chunk::grouped(blockIdx.x, wv, WPG) : blockIdx.x, L, H, C);
  const int m = VARLEN ? ch.m : C;
  if (VARLEN && m <= 0) return;  // the whole workgroup (its waves share the chunk)
  const int64_t tile = ch.tile;
  const GateRows<C> gr = fetch_gates<C>(beta, g, ch, L, H, m);
  const Lane ln = lane_here();

  Pair<F> kp[NB][DK / 32];
  load_rows<NB, DK>(kp, K + ch.row(0, L, H, DK), (int64_t)H * DK, ln, m);
  stash_gates<C, (WPG > 1)>(gr, sb, sg);
  // issued once K has been consumed: the compiler counts DMA completions as
  // unordered with plain loads and would otherwise wait for V before the
  // Gram; the inverse that follows touches no global memory
  auto prefetch_v = [&]() {
    if constexpr (PREF) {
      __builtin_amdgcn_sched_barrier(0);
      prefetch_rows_lds<NB, DV>((const __bf16*)V + ch.row(0, L, H, DV), (int64_t)H * DV, sv, ln, m);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  Acc<NB> Tr;
  chunk_inverse<NB, DK, F, SMALLN, NC, SC, EXACT>(kp, sb, sg, N, S, Tr, prefetch_v);
  if (Tout) store_unit_row<NB>(Tout + tile * (C * C), C, Tr);
#pragma unroll
  for (int I = 0; I < NB; ++I) Tr.a[bidx(I, I)] = band_block<false>(Tr.a[bidx(I, I)], 0, 1, C) + eye4();
  RowP<NB, F> TR;
  scale_cols(TR, Tr, sb);
  // with the prefetch, U is formed first from V read out of LDS one slice at
  // a time, then W from the K pairs, so K and V are never both in registers
  const int64_t ldk = (int64_t)H * DK, ldv = (int64_t)H * DV;
  if constexpr (PREF) {
    wait_vmem();
    apply_lower<NB, DV>(TR, LdsRows<DV>{sv, ln.id}, U + ch.row(0, L, H, DV), ldv, ln, (TIO*)nullptr, m);
    apply_lower<NB, DK>(TR, RegRows<NB, DK, F>{kp}, W + ch.row(0, L, H, DK), ldk, ln, (TIO*)nullptr, m);
  } else if constexpr (NB <= 2) {  // registers to spare: V's loads overlap W
    Pair<F> vp[NB][DV / 32];
    load_rows<NB, DV>(vp, V + ch.row(0, L, H, DV), ldv, ln, m);
    apply_lower<NB, DK>(TR, RegRows<NB, DK, F>{kp}, W + ch.row(0, L, H, DK), ldk, ln, (TIO*)nullptr, m);
    apply_lower<NB, DV>(TR, RegRows<NB, DV, F>{vp}, U + ch.row(0, L, H, DV), ldv, ln, (TIO*)nullptr, m);
  } else {
    apply_lower<NB, DK>(TR, RegRows<NB, DK, F>{kp}, W + ch.row(0, L, H, DK), ldk, ln, (TIO*)nullptr, m);
    Pair<F> vp[NB][DV / 32];
    load_rows<NB, DV>(vp, V + ch.row(0, L, H, DV), ldv, ln, m);
    apply_lower<NB, DV>(TR, RegRows<NB, DV, F>{vp}, U + ch.row(0, L, H, DV), ldv, ln, (TIO*)nullptr, m);
  }
}

// ---------------------------------------------------------------------------
// gdn_chunk_wy_fused at C = 128: the block form of Appendix E with two waves
// per chunk.  With the 64-row halves 1, 2 of the chunk, X_kk the inverses of
// (I + A_kk) by the engine and X_21 = -X_22 A_21 X_11,
//   W_1 = X_11 diag(beta_1) K_1,
//   W_2 = X_21 diag(beta_1) K_1 + X_22 diag(beta_2) K_2,
// and the same for U with V.  Wave 0 inverts its diagonal block, hands X_11
// to wave 1 through LDS and forms W_1, U_1; wave 1 inverts its own block,
// builds A_21 from K_2 and the LDS copy of K_1, then X_21 and W_2, U_2.
// Half 2 never waits for half 1's outputs.  The waves meet at three workgroup
// barriers: both K halves stored; X_11 stored; and, with W_1 and W_2 formed,
// before both read V_1, so that its second read is an L2 hit (wave 0, which
// has less to do, waits there).  Every branch below is uniform per wave.

// A_21 (times `sign`): rows in half 2, columns in half 1, all entries live;
// row form, blocks [I][J]
template <typename F>
__device__ __forceinline__ void gate_rect(f32x4 (&G)[4][4], const float* sb2, const float* sg2,
                                          const float* sg1, float sign, Lane ln) {
  const int g = ln.g(), c = ln.c();
#pragma unroll
  for (int I = 0; I < 4; ++I)
#pragma unroll
    for (int J = 0; J < 4; ++J)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = I * 16 + c, j = J * 16 + 4 * g + v;
        G[I][J][v] = sign * sb2[i] * G[I][J][v] * __expf(sg2[i] - sg1[j]);
      }
}

// out_2 = X21' X_1 + X22' X_2 for the rows of half 2: X21' (all blocks) and
// X22' (lower) as row pairs with beta folded into their columns, X_1 and X_2
// given by get1(I, q) / get2(I, q) as row-form pairs of the two halves, 32
// features at a time; x1, x2 hold slice 0 on entry (the caller may issue its
// loads early).  PIPE: the loads of slice q + 1 go out before the products
// of slice q (two slices of operands live), else each slice is loaded in its
// turn.  Each 16 x 16 block of X is moved to column form by an identity
// MFMA, as in apply_lower; rows at or past m2 are not stored.
template <int D, bool PIPE, typename F, typename TIO, typename Get1, typename Get2>
__device__ __forceinline__ void apply_half2(const RowP<4, F>& X21R, const RowP<4, F>& X22R,
                                            Get1&& get1, Get2&& get2, Pair<F> (&x1)[4],
                                            Pair<F> (&x2)[4], TIO* __restrict__ ob, int64_t ld,
                                            Lane ln, int m2) {
  const int g = ln.g(), c = ln.c();
  const f32x4 e = eye4(ln);
  const Pair<F> id0 = Pair<F>::make(e, zero4()), id1 = Pair<F>::make(zero4(), e);
#pragma unroll
  for (int q = 0; q < D / 32; ++q) {
    if (!PIPE && q > 0) {
#pragma unroll
      for (int I = 0; I < 4; ++I) {
        x1[I] = get1(I, q);
        x2[I] = get2(I, q);
      }
    }
    Pair<F> y1[2][2], y2[2][2];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const Pair<F> id = h ? id1 : id0;
        y1[h][p] = Pair<F>::make(Pair<F>::template mma<false>(x1[2 * p], id, zero4()),
                                 Pair<F>::template mma<false>(x1[2 * p + 1], id, zero4()));
        y2[h][p] = Pair<F>::make(Pair<F>::template mma<false>(x2[2 * p], id, zero4()),
                                 Pair<F>::template mma<false>(x2[2 * p + 1], id, zero4()));
      }
    if (PIPE && q + 1 < D / 32) {
#pragma unroll
      for (int I = 0; I < 4; ++I) {
        x1[I] = get1(I, q + 1);
        x2[I] = get2(I, q + 1);
      }
    }
#pragma unroll
    for (int I = 0; I < 4; ++I) {
      f32x4 acc[2] = {zero4(), zero4()};
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          acc[h] = Pair<F>::template mma<true>(X21R.r[I][p], y1[h][p], acc[h]);
          if (2 * p <= I) acc[h] = Pair<F>::template mma<true>(X22R.r[I][p], y2[h][p], acc[h]);
        }
      if (I * 16 + c < m2) store_row8(ob + (I * 16 + c) * ld + 32 * q + 8 * g, acc[0], acc[1]);
    }
  }
}

// VARLEN: packed sequences (B = 1, L = T tokens, chunk tables pk): a chunk
// of m < 128 tokens is the tile padded with tokens that write nothing (beta
// = 0, keys and values read from the last token and zeroed), so its rows
// past m are neither read for output nor written; a half with no token
// (m <= 64) still runs, on zeros.
// Both K halves stay in LDS (the register copy dies after the Gram product,
// leaving the registers to the inverse); X_11 goes to wave 1 as the six live
// column pairs of its blocks.  GRP > 1 (fixed layout): the workgroup holds
// GRP chunks of neighbouring heads of one chunk row (Chunk::grouped), two
// waves and their own LDS arrays each, so that one CU issues the loads and
// stores of a contiguous run of every token row; the barriers are common.
template <int DK, int DV, typename F, bool SMALLN, int NC, int SC, typename TIO,
          bool EXACT = false, bool VARLEN = false, int GRP = 1>
__global__ __launch_bounds__(128 * GRP) void k_fused128(const TIO* __restrict__ K,
                                                  const TIO* __restrict__ V,
                                                  const float* __restrict__ beta,
                                                  const float* __restrict__ g,
                                                  TIO* __restrict__ W, TIO* __restrict__ U,
                                                  TIO* __restrict__ Tout, int L, int H, int N,
                                                  int S, Packed pk) {
  constexpr int NB = 4, C = 128, KS = NB * (DK / 32) * 512;
  static_assert(!VARLEN || GRP == 1, "packed chunks may end early: one chunk per workgroup");
  __shared__ float sb_[GRP][C], sg_[GRP][C];
  __shared__ __attribute__((aligned(16))) TIO sK_[GRP][2 * KS];  // K_1, K_2 in LdsRows slots
  __shared__ Pair<F> sXc_[GRP][6][64];  // X_11 column pairs (p, J), 2p + 1 >= J
  const int wall = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pi = GRP > 1 ? wall >> 1 : 0;  // this wave's chunk in the workgroup
  const int wv = wall & 1;                 // and its half of that chunk
  float* const sb = sb_[pi];
  float* const sg = sg_[pi];
  TIO* const sK = sK_[pi];
  Pair<F>(&sXc)[6][64] = sXc_[pi];
  Chunk ch;
  if constexpr (VARLEN)
    ch = Chunk::packed(blockIdx.x, H, C, L, pk.cu, pk.off, pk.nseq, pk.nchunks);
  else
    ch = Chunk(GRP > 1 ? Chunk::grouped(blockIdx.x, pi, GRP) : blockIdx.x, L, H, C);
  const int m = VARLEN ? ch.m : C;
  if (VARLEN && m <= 0) return;  // the whole workgroup, before any barrier
  const Lane ln = lane_here();
  const int gq = ln.g(), cq = ln.c();
  const int64_t ldk = (int64_t)H * DK, ldv = (int64_t)H * DV;
  {
    const int r = threadIdx.x & 127;  // 128 threads per chunk, one row each
    const int rr = r < m ? r : m - 1;
    const int64_t o = ((int64_t)ch.b * L + ch.t0 + rr) * H + ch.h;
    sb[r] = r < m ? beta[o] : 0.f;
    sg[r] = g[o];
  }
  // ---- this wave's half: K rows (to LDS), A_kk, X_kk (rows past m read
  // from row m - 1 and zeroed: the base is row r0, so the row count passed is
  // m - r0)
  const int r0 = 64 * wv;
  const LdsRows<DK, F, TIO> k1s{sK, ln.id}, k2s{sK + KS, ln.id};
  Acc<NB> Tr;
  {
    Pair<F> kp[NB][DK / 32];
    load_rows<NB, DK>(kp, K + ch.row(r0, L, H, DK), ldk, ln, m - r0);
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int q = 0; q < DK / 32; ++q)
        store_row8(sK + wv * KS + 512 * (I * (DK / 32) + q) + 8 * ln.id, kp[I][q].lo(),
                   kp[I][q].hi());
    __syncthreads();  // gates and both K halves in LDS
    chunk_inverse<NB, DK, F, SMALLN, NC, SC, EXACT>(kp, sb + r0, sg + r0, N, S, Tr, [] {});
  }
#pragma unroll
  for (int I = 0; I < NB; ++I) Tr.a[bidx(I, I)] = band_block<false>(Tr.a[bidx(I, I)], 0, 1, 64) + eye4();
  Pair<F> NA[4][2];  // wave 1: -A_21, row pairs
  if (wv == 0) {
    // X_11 to LDS in column form
    RowP<NB, F> XR;
    to_rowp(XR, Tr);
    Acc<NB> Xc;
    row_to_col(Xc, XR, 0, 63, ln);
    ColP<NB, F> XC;
    to_colp(XC, Xc);
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int J = 0; J <= 2 * p + 1; ++J) sXc[2 * p + J][ln.id] = XC.c[p][J];
  } else {
    f32x4 G[4][4];
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int J = 0; J < 4; ++J) G[I][J] = zero4();
#pragma unroll
    for (int q = 0; q < DK / 32; ++q) {
      Pair<F> k1[4], k2[4];
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        k1[J] = k1s(J, q);
        k2[J] = k2s(J, q);
      }
#pragma unroll
      for (int I = 0; I < 4; ++I)
#pragma unroll
        for (int J = 0; J < 4; ++J) G[I][J] = Pair<F>::template mma<true>(k2[I], k1[J], G[I][J]);
    }
    gate_rect<F>(G, sb + 64, sg + 64, sg, -1.f, ln);
#pragma unroll
    for (int I = 0; I < 4; ++I)
#pragma unroll
      for (int p = 0; p < 2; ++p) NA[I][p] = Pair<F>::make(G[I][2 * p], G[I][2 * p + 1]);
  }
  __syncthreads();  // X_11 in LDS
  if (wv == 0) {
    // ---- half 1: Tout rows 0..63, then W_1, U_1
    if (Tout) {
      TIO* t = Tout + ch.tile * (C * C);
      store_unit_row<NB>(t, C, Tr);
#pragma unroll
      for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int J = 0; J < NB; ++J) store4(t + (I * 16 + cq) * C + 64 + J * 16 + 4 * gq, zero4());
    }
    RowP<NB, F> TR;
    scale_cols(TR, Tr, sb);
    apply_lower<NB, DK>(TR, k1s, W + ch.row(0, L, H, DK), ldk, ln, (TIO*)nullptr, m);
    __syncthreads();  // wave 1 has formed W_2: both waves read V_1 together
    Pair<F> vp[NB][DV / 32];
    load_rows<NB, DV>(vp, V + ch.row(0, L, H, DV), ldv, ln, m);
    apply_lower<NB, DV>(TR, RegRows<NB, DV, F>{vp}, U + ch.row(0, L, H, DV), ldv, ln,
                        (TIO*)nullptr, m);
  } else {
    // ---- half 2: X_21 = X_22 M with M = -A_21 X_11, one column pair of
    // blocks at a time, then W_2 and U_2
    auto vrow = [&](int base, int I, int q) {
      const int r = base + I * 16 + cq, rr = r < m ? r : m - 1;
      const Pair<F> x = load_row8<F>(V + ch.row(rr, L, H, DV) + 32 * q + 8 * gq);
      return r < m ? x : Pair<F>::zero();
    };
    TIO* const t = Tout ? Tout + ch.tile * (C * C) : nullptr;
    if (t) store_unit_row<NB>(t + 64 * C + 64, C, Tr);
    RowP<4, F> X21R, X22S;  // X_22 diag(beta_2) for the products below
    scale_cols(X22S, Tr, sb + 64);
    {
      RowP<4, F> X22R;
      to_rowp(X22R, Tr);
#pragma unroll
      for (int p2 = 0; p2 < 2; ++p2) {
        f32x4 X21[4][2];
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int J = 2 * p2 + jj;
          f32x4 M[4];
#pragma unroll
          for (int I = 0; I < 4; ++I) {
            f32x4 acc = zero4();
#pragma unroll
            for (int p = 0; p < 2; ++p)
              if (2 * p + 1 >= J)
                acc = Pair<F>::template mma<false>(NA[I][p], sXc[2 * p + J][ln.id], acc);
            M[I] = acc;
          }
          const Pair<F> mc[2] = {Pair<F>::make(M[0], M[1]), Pair<F>::make(M[2], M[3])};
#pragma unroll
          for (int I = 0; I < 4; ++I) {
            f32x4 acc = zero4();
#pragma unroll
            for (int p = 0; p < 2; ++p)
              if (2 * p <= I) acc = Pair<F>::template mma<true>(X22R.r[I][p], mc[p], acc);
            X21[I][jj] = acc;
          }
        }
        if (t) {
#pragma unroll
          for (int I = 0; I < 4; ++I)
#pragma unroll
            for (int jj = 0; jj < 2; ++jj)
              store4(t + (64 + I * 16 + cq) * C + (2 * p2 + jj) * 16 + 4 * gq, X21[I][jj]);
        }
#pragma unroll
        for (int I = 0; I < 4; ++I) {
#pragma unroll
          for (int jj = 0; jj < 2; ++jj)
#pragma unroll
            for (int v = 0; v < 4; ++v) X21[I][jj][v] *= sb[(2 * p2 + jj) * 16 + 4 * gq + v];
          X21R.r[I][p2] = Pair<F>::make(X21[I][0], X21[I][1]);
        }
      }
    }
    {
      Pair<F> k1[4], k2[4];
#pragma unroll
      for (int I = 0; I < 4; ++I) {
        k1[I] = k1s(I, 0);
        k2[I] = k2s(I, 0);
      }
      apply_half2<DK, false, F>(X21R, X22S, k1s, k2s, k1, k2, W + ch.row(64, L, H, DK), ldk, ln, m - 64);
    }
    __syncthreads();  // wave 0 reads V_1 for U_1 alongside (one HBM read)
    Pair<F> v1[4], v2[4];
#pragma unroll
    for (int I = 0; I < 4; ++I) {
      v1[I] = vrow(0, I, 0);
      v2[I] = vrow(64, I, 0);
    }
    // over packed sequences the row guards leave no registers for pipelined
    // slices: there V's slices are loaded in turn
    apply_half2<DV, !VARLEN, F>(
        X21R, X22S, [&](int I, int q) { return vrow(0, I, q); },
        [&](int I, int q) { return vrow(64, I, q); }, v1, v2, U + ch.row(64, L, H, DV), ldv, ln,
        m - 64);
  }
}

// ---------------------------------------------------------------------------
// launchers

template <int NB, typename F, typename TK, typename TA>
static hipError_t run_build_A_nb(const void* K, const float* beta, const float* g, void* A,
                                 int64_t n, int L, int H, int dk, hipStream_t st) {
  GDN_DK_SWITCH(dk, {
    hipLaunchKernelGGL((k_build_A<NB, DK, F, TK, TA>), dim3((unsigned)n), dim3(64), 0, st,
                       (const TK*)K, beta, g, (TA*)A, L, H);
    return hipGetLastError();
  })
  return hipErrorNotSupported;
}

template <typename F, typename TK, typename TA>
static hipError_t run_build_A(const void* K, const float* beta, const float* g, void* A,
                              int64_t n, int L, int H, int dk, int C, hipStream_t st) {
  switch (C) {
    case 16: return run_build_A_nb<1, F, TK, TA>(K, beta, g, A, n, L, H, dk, st);
    case 32: return run_build_A_nb<2, F, TK, TA>(K, beta, g, A, n, L, H, dk, st);
    case 64: return run_build_A_nb<4, F, TK, TA>(K, beta, g, A, n, L, H, dk, st);
    case 128: return run_build_A_nb<8, F, TK, TA>(K, beta, g, A, n, L, H, dk, st);
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

template <int NB, typename F, typename TIO>
static hipError_t run_wy_nb(const void* T, const void* K, const void* V, const float* beta,
                            void* W, void* U, int64_t n, int L, int H, int dk, int dv,
                            hipStream_t st) {
  GDN_DK_SWITCH(dk, GDN_DV_SWITCH(dv, {
    hipLaunchKernelGGL((k_wy<NB, DK, DV, F, TIO>), dim3((unsigned)n), dim3(64), 0, st,
                       (const TIO*)T, (const TIO*)K, (const TIO*)V, beta, (TIO*)W, (TIO*)U, L, H);
    return hipGetLastError();
  }))
  return hipErrorNotSupported;
}

template <typename F, typename TIO>
static hipError_t run_wy(const void* T, const void* K, const void* V, const float* beta,
                         void* W, void* U, int64_t n, int L, int H, int dk, int dv, int C,
                         hipStream_t st) {
  switch (C) {
    case 16: return run_wy_nb<1, F, TIO>(T, K, V, beta, W, U, n, L, H, dk, dv, st);
    case 32: return run_wy_nb<2, F, TIO>(T, K, V, beta, W, U, n, L, H, dk, dv, st);
    case 64: return run_wy_nb<4, F, TIO>(T, K, V, beta, W, U, n, L, H, dk, dv, st);
    case 128: return run_wy_nb<8, F, TIO>(T, K, V, beta, W, U, n, L, H, dk, dv, st);
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

template <int NB> struct FusedOrder;
template <> struct FusedOrder<1> { static constexpr int N = 3, S = 2; };
template <> struct FusedOrder<2> { static constexpr int N = 3, S = 4; };
template <> struct FusedOrder<4> { static constexpr int N = 3, S = 8; };

template <int NB, int DK, int DV, typename F, bool SMALLN, int NC, int SC, typename TIO, bool PREF,
          bool EXACT = false>
static void launch_one(const void* K, const void* V, const float* beta, const float* g, void* W,
                       void* U, void* T, int64_t n, int L, int H, int N, int S, hipStream_t st,
                       const Packed& pk = Packed{}) {
  // workgroups of 4 (or 2) waves on neighbouring heads of one chunk
  const int wpg = waves_per_group(H);
  if (pk.cu && wpg == 4)
    hipLaunchKernelGGL((k_fused<NB, DK, DV, F, SMALLN, NC, SC, TIO, PREF, EXACT, true, 4>),
                       dim3((unsigned)(n / 4)), dim3(256), 0, st, (const TIO*)K, (const TIO*)V,
                       beta, g, (TIO*)W, (TIO*)U, (TIO*)T, L, H, N, S, pk.cu, pk.off, pk.nseq,
                       pk.nchunks);
  else if (pk.cu && wpg == 2)
    hipLaunchKernelGGL((k_fused<NB, DK, DV, F, SMALLN, NC, SC, TIO, PREF, EXACT, true, 2>),
                       dim3((unsigned)(n / 2)), dim3(128), 0, st, (const TIO*)K, (const TIO*)V,
                       beta, g, (TIO*)W, (TIO*)U, (TIO*)T, L, H, N, S, pk.cu, pk.off, pk.nseq,
                       pk.nchunks);
  else if (pk.cu)
    hipLaunchKernelGGL((k_fused<NB, DK, DV, F, SMALLN, NC, SC, TIO, PREF, EXACT, true>),
                       dim3((unsigned)n), dim3(64), 0, st, (const TIO*)K, (const TIO*)V, beta, g,
                       (TIO*)W, (TIO*)U, (TIO*)T, L, H, N, S, pk.cu, pk.off, pk.nseq, pk.nchunks);
  else if (wpg == 4)
    hipLaunchKernelGGL((k_fused<NB, DK, DV, F, SMALLN, NC, SC, TIO, PREF, EXACT, false, 4>),
                       dim3((unsigned)(n / 4)), dim3(256), 0, st, (const TIO*)K, (const TIO*)V,
                       beta, g, (TIO*)W, (TIO*)U, (TIO*)T, L, H, N, S, nullptr, nullptr, 0, 0);
  else if (wpg == 2)
    hipLaunchKernelGGL((k_fused<NB, DK, DV, F, SMALLN, NC, SC, TIO, PREF, EXACT, false, 2>),
                       dim3((unsigned)(n / 2)), dim3(128), 0, st, (const TIO*)K, (const TIO*)V,
                       beta, g, (TIO*)W, (TIO*)U, (TIO*)T, L, H, N, S, nullptr, nullptr, 0, 0);
  else
    hipLaunchKernelGGL((k_fused<NB, DK, DV, F, SMALLN, NC, SC, TIO, PREF, EXACT, false>),
                       dim3((unsigned)n), dim3(64), 0, st, (const TIO*)K, (const TIO*)V, beta, g,
                       (TIO*)W, (TIO*)U, (TIO*)T, L, H, N, S, nullptr, nullptr, 0, 0);
}

// bf16 with C >= 32 prefetches V (for C = 16 the tile is small and the
// kernel runs at high occupancy without it)
template <int NB, typename F, typename TIO>
static hipError_t run_fused_nb(const void* K, const void* V, const float* beta, const float* g,
                               void* W, void* U, void* T, int64_t n, int L, int H, int dk,
                               int dv, int N, int S, bool exact, hipStream_t st,
                               const Packed& pk = Packed{}) {
  constexpr int DN = FusedOrder<NB>::N, DS = FusedOrder<NB>::S;
  constexpr bool PREF = sizeof(TIO) == 2 && NB > 1;
  GDN_DK_SWITCH(dk, GDN_DV_SWITCH(dv, {
    if (exact)
      launch_one<NB, DK, DV, F, true, 0, 0, TIO, PREF, true>(K, V, beta, g, W, U, T, n, L, H, N,
                                                             S, st, pk);
    else if (N == DN && S == DS)
      launch_one<NB, DK, DV, F, true, DN, DS, TIO, PREF>(K, V, beta, g, W, U, T, n, L, H, N, S,
                                                          st, pk);
    else if (N <= 15)
      launch_one<NB, DK, DV, F, true, -1, -1, TIO, PREF>(K, V, beta, g, W, U, T, n, L, H, N, S,
                                                          st, pk);
    else
      launch_one<NB, DK, DV, F, false, -1, -1, TIO, PREF>(K, V, beta, g, W, U, T, n, L, H, N, S,
                                                           st, pk);
    return hipGetLastError();
  }))
  return hipErrorNotSupported;
}

template <typename F, typename TIO>
static hipError_t run_fused128(const void* K, const void* V, const float* beta, const float* g,
                               void* W, void* U, void* T, int64_t n, int L, int H, int dk,
                               int dv, int N, int S, bool exact, hipStream_t st,
                               const Packed& pk = Packed{}) {
  // fixed layout: two chunks of neighbouring heads per workgroup
  // (Chunk::grouped) when 16 divides H
  constexpr int GRPN = 2;
  const bool grp = H % (8 * GRPN) == 0;
#define GDN_F128_(SM, NC_, SC_, EX, VL, G)                                                       \
  hipLaunchKernelGGL((k_fused128<DK, DV, F, SM, NC_, SC_, TIO, EX, VL, G>), dim3((unsigned)(n / G)), \
                     dim3(128 * G), 0, st, (const TIO*)K, (const TIO*)V, beta, g, (TIO*)W,        \
                     (TIO*)U, (TIO*)T, L, H, N, S, pk)
#define GDN_F128(SM, NC_, SC_, EX)          \
  if (pk.cu)                                \
    GDN_F128_(SM, NC_, SC_, EX, true, 1);    \
  else if (grp)                             \
    GDN_F128_(SM, NC_, SC_, EX, false, GRPN); \
  else                                      \
    GDN_F128_(SM, NC_, SC_, EX, false, 1)
  GDN_DK_SWITCH(dk, GDN_DV_SWITCH(dv, {
    if (exact)
      GDN_F128(true, 0, 0, true);
    else if (N == 3 && S == 8)
      GDN_F128(true, 3, 8, false);
    else if (N <= 15)
      GDN_F128(true, -1, -1, false);
    else
      GDN_F128(false, -1, -1, false);
    return hipGetLastError();
  }))
#undef GDN_F128
#undef GDN_F128_
  return hipErrorNotSupported;
}

template <typename F, typename TIO>
static hipError_t run_fused(const void* K, const void* V, const float* beta, const float* g,
                            void* W, void* U, void* T, int64_t n, int L, int H, int dk, int dv,
                            int C, int N, int S, bool exact, hipStream_t st) {
  switch (C) {
    case 128: return run_fused128<F, TIO>(K, V, beta, g, W, U, T, n, L, H, dk, dv, N, S, exact, st);
    case 16: return run_fused_nb<1, F, TIO>(K, V, beta, g, W, U, T, n, L, H, dk, dv, N, S, exact, st);
    case 32: return run_fused_nb<2, F, TIO>(K, V, beta, g, W, U, T, n, L, H, dk, dv, N, S, exact, st);
    case 64: return run_fused_nb<4, F, TIO>(K, V, beta, g, W, U, T, n, L, H, dk, dv, N, S, exact, st);
  }
  return hipErrorNotSupported;
}

hipError_t launch_fused_varlen(const void* K, const void* V, const float* beta, const float* g,
                               void* W, void* U, void* T, const int* cu, const int* off, int nseq,
                               int nchunks, int Ttok, int H, int dk, int dv, int C, int N, int S,
                               int dtype, bool exact, hipStream_t st) {
  const Packed pk{cu, off, nseq, nchunks};
  const int64_t n = (int64_t)nchunks * H;
#define GDN_FV(NB_, F_, T_)                                                                     \
  return run_fused_nb<NB_, F_, T_>(K, V, beta, g, W, U, T, n, Ttok, H, dk, dv, N, S, exact, st, \
                                   pk)
  if (dtype == 0) {
    switch (C) {
      case 16: GDN_FV(1, f32x4, float);
      case 32: GDN_FV(2, f32x4, float);
      case 64: GDN_FV(4, f32x4, float);
      case 128:
        return run_fused128<f32x4, float>(K, V, beta, g, W, U, T, n, Ttok, H, dk, dv, N, S, exact,
                                          st, pk);
    }
  } else if (dtype == 1) {
    switch (C) {
      case 16: GDN_FV(1, bf16x4, __bf16);
      case 32: GDN_FV(2, bf16x4, __bf16);
      case 64: GDN_FV(4, bf16x4, __bf16);
      case 128:
        return run_fused128<bf16x4, __bf16>(K, V, beta, g, W, U, T, n, Ttok, H, dk, dv, N, S,
                                            exact, st, pk);
    }
  }
#undef GDN_FV
  return hipErrorNotSupported;
}

hipError_t launch_fused(const void* K, const void* V, const float* beta, const float* g, void* W,
                        void* U, void* T, int B, int L, int H, int dk, int dv, int C, int N,
                        int S, int dtype, bool exact, hipStream_t st) {
  const int64_t n = (int64_t)B * H * (L / C);
  if (dtype == 0)
    return run_fused<f32x4, float>(K, V, beta, g, W, U, T, n, L, H, dk, dv, C, N, S, exact, st);
  if (dtype == 1)
    return run_fused<bf16x4, __bf16>(K, V, beta, g, W, U, T, n, L, H, dk, dv, C, N, S, exact, st);
  return hipErrorNotSupported;
}

}  // namespace gdn
