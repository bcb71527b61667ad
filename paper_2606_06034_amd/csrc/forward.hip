// forward.hip -- the chunk-wise Gated DeltaNet forward around the chunk
// inverse: per chunk the WY factors, then the state recurrence across the
// chunks of a head and the output (the chunk-level recurrence of Gated
// DeltaNet that Section 1 builds on; Y = T^-1 X of Appendix E).
//
// With gamma the within-chunk cumulative log-decay (the g input), per chunk
//   T = (I + A)^-1,  W = T diag(beta e^gamma) K,  U = T diag(beta) V,
//   P = (Q K^T) (.) D,  D_ij = e^{gamma_i - gamma_j} for i >= j, else 0,
// and across chunks, with S the [dk, dv] state entering the chunk,
//   V_new = U - W S,
//   O     = scale (diag(e^gamma) Q S + P V_new),
//   S'    = e^{gamma_last} S + K^T diag(e^{gamma_last - gamma}) V_new.
//
// Stage 1, k_fwd_chunk: one wave per chunk, every chunk in parallel.  Forms
// T (Neumann engine or exact block-wise inverse), then W, U, K^T and P, and
// stores them in the workspace in exactly the register-fragment layouts
// stage 2 feeds to its MFMAs, so stage 2 reads each operand with one 16-byte
// load per lane from a contiguous 1 KB run per wave and changes no layout.
// Stage 2, k_fwd_state: one workgroup per (batch, head, 16 value columns).
// It walks the chunks of its head in order with its dk x 16 slice of S in
// registers (fp32), spread over four waves; per chunk four product groups:
// W S, Q S, P V_new and K^T V_new.
//
// Fragment conventions (tile16.hpp): a pair over 16-blocks {2p, 2p + 1}
// gives slot s of lane (g, c) the index 32p + 16 (s / 4) + 4g + s % 4; a
// pair loaded as a run of 8 features gives slot s the feature 32q + 8g + s.
// The 16 value columns of slice j = 2jq + jh are, for block column n,
//   dv(n) = 32 jq + 8 (n / 4) + 4 jh + n % 4
// (the column order the identity-MFMA transposes of a 32-feature run
// produce), and state block m = 2q' + h' holds, for block row r = 4g + v,
//   dk = 32 q' + 8 g + 4 h' + v,
// so that the pair (block 2q', block 2q' + 1) lines up with a run of 8
// features of W and Q rows.
#include <mutex>
#include <type_traits>

#include "int16_ops.hpp"
#include "int8_ops.hpp"
#include "launch.hpp"
#include "wy.hpp"

namespace gdn {

// Workspace parts per chunk tile, in elements of the IO type.  A slot is one
// pair per lane (64 x 8 elements); a column-form block 64 x 4.
//   W : NB x (DK / 32) slots, W row pairs (I, q)
//   U : (DV / 16) x NB blocks, U column blocks (slice j, I)
//   KT: (DK / 16) x npair(NB) slots, K^T row pairs (state block m, p)
//   P : npp(NB) slots, P row pairs (I, p) with 2p <= I
__host__ __device__ constexpr int npp(int NB) {
  int n = 0;
  for (int I = 0; I < NB; ++I) n += I / 2 + 1;
  return n;
}
// sum over i < I of (i / 2 + 1), in closed form (I may be a runtime value)
__host__ __device__ constexpr int pidx(int I, int p) {
  return I + (I / 2) * ((I - 1) / 2) + p;
}
template <int NB, int DK, int DV>
struct FwdLayout {
  static constexpr int64_t W = NB * (DK / 32) * 512;
  static constexpr int64_t U = (DV / 16) * NB * 256;
  static constexpr int64_t KT = (DK / 16) * npair(NB) * 512;
  static constexpr int64_t P = npp(NB) * 512;
  static constexpr int64_t tile = W + U + KT + P;
};

int64_t fwd_workspace_elems(int C, int dk, int dv) {
  const int NB = C / 16, np = (NB + 1) / 2;
  return (int64_t)NB * (dk / 32) * 512 + (int64_t)(dv / 16) * NB * 256 +
         (int64_t)(dk / 16) * np * 512 + (int64_t)npp(NB) * 512;
}

// One fragment slot: a pair per lane, 64 x 8 values.  bf16: lane-major runs
// of 8 (16 bytes per lane); fp32: the lo halves of all lanes, then the hi
// halves (16 bytes per lane each), so that every slot is a whole number of
// 1 KB runs of 16 bytes per lane, the unit of a wave's global -> LDS copy.
__device__ __forceinline__ void slot_store(__bf16* s, const Pair<bf16x4>& x, int l) {
  *(bf16x8*)(s + 8 * l) = x.v;
}
__device__ __forceinline__ void slot_store(float* s, const Pair<f32x4>& x, int l) {
  *(f32x4*)(s + 4 * l) = x.a;
  *(f32x4*)(s + 256 + 4 * l) = x.b;
}
__device__ __forceinline__ void slot_store(__bf16* s, f32x4 lo, f32x4 hi, int l) {
  store_row8(s + 8 * l, lo, hi);
}
__device__ __forceinline__ void slot_store(float* s, f32x4 lo, f32x4 hi, int l) {
  *(f32x4*)(s + 4 * l) = lo;
  *(f32x4*)(s + 256 + 4 * l) = hi;
}
template <typename F, typename TIO>
__device__ __forceinline__ Pair<F> slot_load(const TIO* s, int l);
template <>
__device__ __forceinline__ Pair<bf16x4> slot_load<bf16x4, __bf16>(const __bf16* s, int l) {
  return Pair<bf16x4>{*(const bf16x8*)(s + 8 * l)};
}
template <>
__device__ __forceinline__ Pair<f32x4> slot_load<f32x4, float>(const float* s, int l) {
  return Pair<f32x4>{*(const f32x4*)(s + 4 * l), *(const f32x4*)(s + 256 + 4 * l)};
}

// Column-form blocks of a 32-feature run of X (rows of the chunk), made by
// identity MFMAs: y[h][p] pairs t-blocks {2p, 2p + 1}; column n of half h is
// feature 32q + 8 (n / 4) + 4h + n % 4.
template <int NB, typename F>
__device__ __forceinline__ void run_to_cols(Pair<F> (&y)[2][npair(NB)], const Pair<F> (&x)[NB],
                                            Lane ln) {
  const f32x4 e = eye4(ln);
  const Pair<F> id0 = Pair<F>::make(e, zero4()), id1 = Pair<F>::make(zero4(), e);
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
}

// U = T' V (T' = T diag(beta) as row pairs) as column-form blocks per
// 16-column slice, from the row pairs of V given by get(I, q).
template <int NB, int DV, typename F, typename TIO, typename Get>
__device__ __forceinline__ void apply_u_fwd(const RowP<NB, F>& TR, Get&& get,
                                            TIO* __restrict__ uf, Lane ln) {
#pragma unroll
  for (int q = 0; q < DV / 32; ++q) {
    Pair<F> x[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) x[I] = get(I, q);
    Pair<F> y[2][npair(NB)];
    run_to_cols<NB, F>(y, x, ln);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int I = 0; I < NB; ++I) {
        f32x4 acc = zero4();
#pragma unroll
        for (int p = 0; p < npair(NB); ++p)
          if (2 * p <= I) acc = Pair<F>::template mma<false>(TR.r[I][p], y[h][p], acc);
        store4(uf + ((2 * q + h) * NB + I) * 256 + 4 * ln.id, acc);
      }
  }
}

// W = T'' K (T'' = T diag(beta e^gamma)) as row pairs over runs of 8
// features, and the column-form blocks of K (= row pairs of K^T) on the way.
template <int NB, int DK, typename F, typename TIO>
__device__ __forceinline__ void apply_w_fwd(const RowP<NB, F>& TR,
                                            const Pair<F> (&kp)[NB][DK / 32],
                                            TIO* __restrict__ wf, TIO* __restrict__ ktf, Lane ln) {
  constexpr int NP = npair(NB);
#pragma unroll
  for (int q = 0; q < DK / 32; ++q) {
    Pair<F> x[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) x[I] = kp[I][q];
    Pair<F> y[2][NP];
    run_to_cols<NB, F>(y, x, ln);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int p = 0; p < NP; ++p) slot_store(ktf + ((2 * q + h) * NP + p) * 512, y[h][p], ln.id);
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      f32x4 acc[2] = {zero4(), zero4()};
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int p = 0; p < NP; ++p)
          if (2 * p <= I) acc[h] = Pair<F>::template mma<true>(TR.r[I][p], y[h][p], acc[h]);
      slot_store(wf + (I * (DK / 32) + q) * 512, acc[0], acc[1], ln.id);
    }
  }
}

// ---------------------------------------------------------------------------
// stage 1

// The inverse modes of the per-chunk launch: T_hat(N, S) in the compute
// type, the exact block-wise inverse, or T_hat(N, S) in integer arithmetic
// (16- or 8-bit codes).
enum FwdInv { kInvNeumann = 0, kInvExact = 1, kInvInt16 = 2, kInvInt8 = 3 };

// The integer inverse of one chunk inside the layer (the quantised GDN of
// Section 3.5): A in fp32 from the K row pairs with the Gram products and
// gates of gdn_build_A, quantised per tile by the quantiser's rule, the
// integer T_hat(N, S) of the shared engine, and its strict lower part
// dequantised (codes * 2^e, exact in fp32) in row form; the caller adds I.
// The codes equal those of gdn_chunk_inverse_neumann_i16_fused (_i8_fused)
// for the same chunk.
template <int NB, int DK, typename F, int INV, int NC, int SC, typename Hook>
__device__ __forceinline__ void chunk_inverse_int(const Pair<F> (&kp)[NB][DK / 32],
                                                  const float* sb, const float* sg, int N, int S,
                                                  Acc<NB>& Tr, Hook&& after_gram) {
  Acc<NB> G;
  gram_lower<NB, DK, true>(G, kp);
  after_gram();
  gate_scale<NB, true>(G, sb, sg, 1.f);
  float m = 0.f;
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) m = fmaxf(m, fabsf(G.a[b][v]));
  const float amax =
      __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(__ockl_wfred_max_f32(m))));
  const int e = INV == kInvInt16 ? i16::quant_exp(amax) : i8::quant_exp(amax);
  iq::AccI<NB> Lr;
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) Lr.a[b][v] = -(int)rintf(ldexpf(G.a[b][v], -e));
  iq::AccI<NB> Ti;
  int eT;
  if constexpr (INV == kInvInt16)
    iq::int_engine<i16::I16Ops, NB, false, NC, SC>(Lr, e, N, S, Ti, eT);
  else
    iq::int_engine<i8::I8Ops, NB, false, NC, SC>(Lr, e, N, S, Ti, eT);
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) Tr.a[b][v] = ldexpf((float)Ti.a[b][v], eT);
}

// VARLEN: packed sequences (B = 1, L = T tokens, chunk tables pk); a chunk's
// rows past its m tokens are read from row m - 1 and carry beta = 0, so W, U
// and K^T vanish there (T is the identity on them) and the state pass never
// stores their outputs.
template <int NB, int DK, int DV, typename F, bool SMALLN, int NC, int SC, typename TIO,
          int INV, bool VARLEN = false>
__global__ __launch_bounds__(64) void k_fwd_chunk(const TIO* __restrict__ Q,
                                                  const TIO* __restrict__ K,
                                                  const TIO* __restrict__ V,
                                                  const float* __restrict__ beta,
                                                  const float* __restrict__ g,
                                                  TIO* __restrict__ ws, int64_t n_tiles, int L,
                                                  int H, int N, int S, Packed pk) {
  constexpr int C = 16 * NB;
  constexpr int DMAX = DK > DV ? DK : DV;
  // bf16: V, then Q, arrive in LDS by DMA while registers are busy
  constexpr bool PREF = sizeof(TIO) == 2;
  using LY = FwdLayout<NB, DK, DV>;
  __shared__ float sb[C], sg[C], sbw[C];
  __shared__ __attribute__((aligned(16))) __bf16 sx[PREF ? NB * (DMAX / 32) * 512 : 8];
  Chunk ch;
  if constexpr (VARLEN)
    ch = Chunk::packed(blockIdx.x, H, C, L, pk.cu, pk.off, pk.nseq, pk.nchunks);
  else
    ch = Chunk(blockIdx.x, L, H, C);
  const int m = VARLEN ? ch.m : C;
  if (VARLEN && m <= 0) return;
  const Lane ln = lane_here();
  const GateRows<C> gr = fetch_gates<C>(beta, g, ch, L, H, m);
  TIO* wf = ws + ch.tile * LY::W;
  TIO* uf = ws + n_tiles * LY::W + ch.tile * LY::U;
  TIO* ktf = ws + n_tiles * (LY::W + LY::U) + ch.tile * LY::KT;
  TIO* pf = ws + n_tiles * (LY::W + LY::U + LY::KT) + ch.tile * LY::P;
  const int64_t ldk = (int64_t)H * DK, ldv = (int64_t)H * DV;

  Pair<F> kp[NB][DK / 32];
  load_rows<NB, DK>(kp, K + ch.row(0, L, H, DK), ldk, ln, m);
  stash_gates<C>(gr, sb, sg);
  for (int r = ln.id; r < C; r += 64) sbw[r] = sb[r] * __expf(sg[r]);
  __syncthreads();
  auto prefetch_v = [&]() {
    if constexpr (PREF) {
      __builtin_amdgcn_sched_barrier(0);
      prefetch_rows_lds<NB, DV>((const __bf16*)V + ch.row(0, L, H, DV), ldv, sx, ln, m);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  Acc<NB> Tr;
  if constexpr (INV == kInvInt16 || INV == kInvInt8)
    chunk_inverse_int<NB, DK, F, INV, NC, SC>(kp, sb, sg, N, S, Tr, prefetch_v);
  else
    chunk_inverse<NB, DK, F, SMALLN, NC, SC, INV == kInvExact>(kp, sb, sg, N, S, Tr, prefetch_v);
#pragma unroll
  for (int I = 0; I < NB; ++I) Tr.a[bidx(I, I)] = band_block<false>(Tr.a[bidx(I, I)], 0, 1, C) + eye4();

  RowP<NB, F> TR;
  scale_cols(TR, Tr, sb);
  if constexpr (PREF) {
    wait_vmem();
    apply_u_fwd<NB, DV, F>(TR, LdsRows<DV>{sx, ln.id}, uf, ln);
    // Q replaces V in LDS: every read of V above has returned its data
    __builtin_amdgcn_sched_barrier(0);
    prefetch_rows_lds<NB, DK>((const __bf16*)Q + ch.row(0, L, H, DK), ldk, sx, ln, m);
    __builtin_amdgcn_sched_barrier(0);
  } else {
    Pair<F> vp[NB][DV / 32];
    load_rows<NB, DV>(vp, V + ch.row(0, L, H, DV), ldv, ln, m);
    apply_u_fwd<NB, DV, F>(TR, RegRows<NB, DV, F>{vp}, uf, ln);
  }
  scale_cols(TR, Tr, sbw);
  apply_w_fwd<NB, DK, F>(TR, kp, wf, ktf, ln);

  // P = (Q K^T) (.) D, lower blocks in row form
  Acc<NB> Pm;
#pragma unroll
  for (int b = 0; b < nlower(NB); ++b) Pm.a[b] = zero4();
  if constexpr (PREF) wait_vmem();
#pragma unroll
  for (int q = 0; q < DK / 32; ++q) {
    Pair<F> qp[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      if constexpr (PREF)
        qp[I] = LdsRows<DK>{sx, ln.id}(I, q);
      else
        qp[I] = load_row8<F>(Q + ch.row(min(I * 16 + ln.c(), m - 1), L, H, DK) + 32 * q +
                             8 * ln.g());
    }
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int J = 0; J <= I; ++J)
        Pm.a[bidx(I, J)] = Pair<F>::template mma<true>(qp[I], kp[J][q], Pm.a[bidx(I, J)]);
  }
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = 0; J <= I; ++J)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = I * 16 + ln.c(), j = J * 16 + 4 * ln.g() + v;
        const float x = Pm.a[bidx(I, J)][v];
        Pm.a[bidx(I, J)][v] = (i >= j) ? x * __expf(sg[i] - sg[j]) : 0.f;
      }
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int p = 0; 2 * p <= I; ++p)
      slot_store(pf + pidx(I, p) * 512, Pair<F>::make(blk(Pm, I, 2 * p), blk(Pm, I, 2 * p + 1)),
                 ln.id);
}

// ---------------------------------------------------------------------------
// stage 2
//
// One workgroup of four waves per (batch, head, slice of 16 value columns),
// one wave per SIMD.  The chunk's work is split so that no wave reads more
// than a quarter of the chunk's operands:
//   wave w owns the state pair q = w (its 2 x 16 state rows) and updates it
//     with K^T rows of those state blocks;
//   wave w forms V_new and O for the row block I = w of the chunk.
// Two small LDS exchanges per chunk connect them: every wave publishes its
// state pair (bf16) before W S and Q S, and its V_new rows (bf16, plain and
// decayed to the chunk end) before P V_new and the state update.  Each
// wave's operands (W, Q, K^T, P rows, U block, gates) come straight from
// global memory into registers, issued DEPTH - 1 chunks ahead into a ring
// of register buffers, so the loads of a chunk overlap the compute of the
// chunks before it.

template <int NB, int DK, typename F>
struct FwdOps {  // one wave's operands of one chunk
  static constexpr int NQ = DK / 32, NP = npair(NB);
  Pair<F> w[NQ];      // W row pairs (I, q)
  Pair<F> q[NQ];      // Q row pairs (I, q)
  Pair<F> kt[2][NP];  // K^T pairs of the owned state blocks
  Pair<F> p[2];       // P row pairs (I, p), p <= I / 2
  f32x4 u;            // U block (slice, I), column form
  float gam;          // gamma of chunk row `lane` (lanes past the chunk's tokens: its last)
};

// half `hf` (block 2p + hf) of slot p
__device__ __forceinline__ void slot_store_half(__bf16* s, f32x4 x, int hf, int l) {
  *(bf16x4*)(s + 8 * l + 4 * hf) = __builtin_convertvector(x, bf16x4);
}
__device__ __forceinline__ void slot_store_half(float* s, f32x4 x, int hf, int l) {
  *(f32x4*)(s + 256 * hf + 4 * l) = x;
}

// VARLEN: one state per (packed sequence, head); the sequence's chunks in
// order, their tiles at h * nchunks + chunk; rows of a chunk past its m
// tokens are read from row m - 1 (Q, g) and not stored (O).  Tables that do
// not describe chunks of C tokens inside the T tokens and nchunks tiles make
// the sequence empty (its final state is its initial one).
template <int NB, int DK, int DV, typename F, typename TIO, int DEPTH, bool VARLEN = false>
__global__ __launch_bounds__(256) void k_fwd_state(const TIO* __restrict__ ws,
                                                   const TIO* __restrict__ Q,
                                                   const float* __restrict__ g,
                                                   const float* __restrict__ S0,
                                                   TIO* __restrict__ O, float* __restrict__ Sfin,
                                                   int64_t n_tiles, int B, int L, int H,
                                                   float scale, Packed pk) {
  constexpr int C = 16 * NB, NQ = DK / 32, NP = npair(NB), NS = DV / 16;
  // DEPTH: chunks whose operands are in registers at once (a ring of
  // buffers, loads issued DEPTH - 1 chunks ahead)
  using LY = FwdLayout<NB, DK, DV>;
  using Ops = FwdOps<NB, DK, F>;
  __shared__ __attribute__((aligned(16))) TIO xs[2][NQ * 512];      // state pairs
  __shared__ __attribute__((aligned(16))) TIO xv[2][2 * NP * 512];  // V_new, V_d pairs
  const int BH = VARLEN ? pk.nseq * H : B * H;
  // work item -> (head bh = b H + h, slice j); when BH is a multiple of 8 the
  // slices of one head share an XCD (work items are dealt to the 8 XCDs in
  // turn), so the rows of W, K^T, P and Q all of them read meet in one L2
  const uint32_t x = blockIdx.x;
  int bh, j;
  if (BH % 8 == 0) {
    const uint32_t r = x >> 3;
    j = (int)(r % NS);
    bh = (int)((r / NS) * 8 + (x & 7));
  } else {
    bh = (int)(x / NS);
    j = (int)(x % NS);
  }
  const int b = bh / H, h = bh - b * H;  // b: the sequence when VARLEN
  // this head's chunks: c0 .. c0 + nc - 1, the first at token tokS; len tokens
  int nc = L / C, c0 = 0, len = L;
  int64_t tokS = (int64_t)b * L;
  if constexpr (VARLEN) {
    const int t0 = pk.cu[b], t1 = pk.cu[b + 1], o0 = pk.off[b], o1 = pk.off[b + 1];
    len = t1 - t0;
    nc = o1 - o0;
    c0 = o0;
    tokS = t0;
    const bool ok = t0 >= 0 && len >= 0 && t1 <= L && o0 >= 0 && nc >= 0 && o1 <= pk.nchunks &&
                    nc == (len + C - 1) / C;
    if (!ok) nc = 0;
  }
  // tokens of chunk ck (C, or fewer in a sequence's last chunk)
  auto rows_of = [&](int ck) { return VARLEN ? min(C, len - ck * C) : C; };
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const Lane ln = lane_here();
  const int l = ln.id, gq = ln.g(), c = ln.c();
  // roles of this wave (uniform; every wave has both at C = 64, dk = 128)
  const bool rows = NB >= 4 || wv < NB, owner = NQ >= 4 || wv < NQ;
  const int jq = j >> 1, jh = j & 1;
  const int dvcol = 32 * jq + 8 * (c >> 2) + 4 * jh + (c & 3);  // column c of the slice
  const int ocol = 32 * jq + 8 * gq + 4 * jh;                   // columns 4g .. 4g + 3
  const int64_t sbase = (int64_t)bh * DK * DV;
  const int64_t ldq = (int64_t)H * DK, ldo = (int64_t)H * DV;
  const TIO* wsW = ws;
  const TIO* wsU = ws + n_tiles * LY::W;
  const TIO* wsKT = wsU + n_tiles * LY::U;
  const TIO* wsP = wsKT + n_tiles * LY::KT;

  // the owned state blocks m = 2 wv, 2 wv + 1: rows dk = 32 wv + 8g + 4 hf + v
  f32x4 st[2] = {zero4(), zero4()};
  if (owner && S0) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        st[hf][v] = S0[sbase + (int64_t)(32 * wv + 8 * gq + 4 * hf + v) * DV + dvcol];
  }
  wait_vmem();  // the initial state is in registers before the loop starts
  if (NB == 1) {  // block 1 of the V_new pair does not exist: zero halves
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
      for (int i = 0; i < 2; ++i) slot_store_half(xv[k] + i * NP * 512, zero4(), 1, l);
  }

  // loads of one chunk's operands in three parts (issued at three points of
  // a step, so no wave stalls on a long burst of loads)
  auto tile_of = [&](int ck) {
    return VARLEN ? (int64_t)h * pk.nchunks + c0 + ck : (int64_t)bh * nc + ck;
  };
  auto load_part = [&](Ops& op, int ck, int part) {
    const int64_t tile = tile_of(ck);
    const int64_t tok0 = tokS + (int64_t)ck * C;
    const int m = rows_of(ck);
    if (part == 0 && rows) {
      const int I = wv;
      const int r = min(I * 16 + c, m - 1);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        op.w[q] = slot_load<F>(wsW + tile * LY::W + (I * NQ + q) * 512, l);
        op.q[q] = load_row8<F>(Q + (tok0 + r) * ldq + (int64_t)h * DK + 32 * q + 8 * gq);
      }
    }
    if (part == 1 && owner) {
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int p = 0; p < NP; ++p)
          op.kt[hf][p] = slot_load<F>(wsKT + tile * LY::KT + ((2 * wv + hf) * NP + p) * 512, l);
    }
    if (part == 2) {
      if (rows) {
        const int I = wv;
#pragma unroll
        for (int p = 0; p < 2; ++p)
          if (2 * p <= I) op.p[p] = slot_load<F>(wsP + tile * LY::P + pidx(I, p) * 512, l);
        op.u = load4(wsU + tile * LY::U + (j * NB + I) * 256 + 4 * l);
      }
      // the chunk's gates in one load, one row per lane; lanes take the
      // rows they need from each other (ds_bpermute)
      op.gam = g[(tok0 + min(l, m - 1)) * H + h];
    }
  };
  auto load = [&](Ops& op, int ck) {
    load_part(op, ck, 0);
    load_part(op, ck, 1);
    load_part(op, ck, 2);
  };

  // one chunk; `nx`, chunk `cknx`: the buffer refilled meanwhile (a
  // compile-time flag, so the loads carry no branches that would blur the
  // compiler's count of loads in flight)
  auto compute = [&](const Ops& op, int ck, Ops& nx, int cknx, auto refill_tag) {
    constexpr bool refill = decltype(refill_tag)::value;
    const int par = ck & 1;
    const int64_t tok0 = tokS + (int64_t)ck * C;
    if (owner) slot_store(xs[par] + wv * 512, Pair<F>::make(st[0], st[1]), l);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (refill) load_part(nx, cknx, 0);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();  // state pairs published
    f32x4 o = zero4();
    const float gl = __builtin_bit_cast(
        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, op.gam), C - 1));
    if (rows) {
      const int I = wv;
      Pair<F> sp[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) sp[q] = slot_load<F>(xs[par] + q * 512, l);
      f32x4 wsum = zero4();
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        wsum = Pair<F>::template mma<false>(op.w[q], sp[q], wsum);
        o = Pair<F>::template mma<true>(op.q[q], sp[q], o);
      }
      const f32x4 vn = op.u - wsum;  // V_new rows 16 I + 4g + v, column form
      f32x4 vd;
#pragma unroll
      for (int v = 0; v < 4; ++v) vd[v] = vn[v] * __expf(gl - __shfl(op.gam, I * 16 + 4 * gq + v));
      slot_store_half(xv[par] + (I >> 1) * 512, vn, I & 1, l);
      slot_store_half(xv[par] + (NP + (I >> 1)) * 512, vd, I & 1, l);
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (refill) load_part(nx, cknx, 1);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();  // V_new published
    if (owner) {
      const float el = __expf(gl);
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        f32x4 acc = el * st[hf];
#pragma unroll
        for (int p = 0; p < NP; ++p)
          acc = Pair<F>::template mma<false>(op.kt[hf][p],
                                             slot_load<F>(xv[par] + (NP + p) * 512, l), acc);
        st[hf] = acc;
      }
    }
    if (rows) {
      const int I = wv;
      o *= __expf(__shfl(op.gam, I * 16 + c));
#pragma unroll
      for (int p = 0; p < 2; ++p)
        if (2 * p <= I)
          o = Pair<F>::template mma<true>(op.p[p], slot_load<F>(xv[par] + p * 512, l), o);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (refill) load_part(nx, cknx, 2);
      __builtin_amdgcn_sched_barrier(0);
      if (!VARLEN || I * 16 + c < rows_of(ck))
        store4(O + (tok0 + I * 16 + c) * ldo + (int64_t)h * DV + ocol, scale * o);
    } else if constexpr (refill) {
      load_part(nx, cknx, 2);
    }
  };
  using Refill = std::integral_constant<bool, true>;
  using NoRefill = std::integral_constant<bool, false>;

  if constexpr (DEPTH == 3) {
    // ring r0, r1, r2: while chunk ck computes from one buffer, the buffer
    // freed by chunk ck - 1 is refilled with chunk ck + 2.  Chunk indices
    // of loads are clamped to the last chunk (a repeated load past the end
    // is harmless), which keeps the loads free of branches
    const int last = nc - 1;
    Ops r0, r1, r2;
    if (nc > 0) {
      load(r0, 0);
      load(r1, min(1, last));
    }
    for (int ck = 0; ck < nc; ck += 3) {
      compute(r0, ck, r2, min(ck + 2, last), Refill{});
      if (ck + 1 >= nc) break;
      compute(r1, ck + 1, r0, min(ck + 3, last), Refill{});
      if (ck + 2 >= nc) break;
      compute(r2, ck + 2, r1, min(ck + 4, last), Refill{});
    }
  } else if constexpr (DEPTH == 2) {
    const int last = nc - 1;
    Ops r0, r1;
    if (nc > 0) load(r0, 0);
    for (int ck = 0; ck < nc; ck += 2) {
      compute(r0, ck, r1, min(ck + 1, last), Refill{});
      if (ck + 1 >= nc) break;
      compute(r1, ck + 1, r0, min(ck + 2, last), Refill{});
    }
  } else {
    for (int ck = 0; ck < nc; ++ck) {
      Ops r, unused;
      load(r, ck);
      compute(r, ck, unused, 0, NoRefill{});
    }
  }
  if (owner && Sfin) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        Sfin[sbase + (int64_t)(32 * wv + 8 * gq + 4 * hf + v) * DV + dvcol] = st[hf][v];
  }
}

// ---------------------------------------------------------------------------
// The scratch of the allocation-free layer forward (gdn_chunk_forward_noalloc):
// the workspace between the two launches, held in a file-scope device array
// of kForwardScratchBytes that every device the library runs on keeps until
// the process ends.  In host code the array's name is only a stand-in for
// its device address: forward_scratch() looks that address up once per
// device (hipGetSymbolAddress with the device current) and hands it out, and
// only that address is ever passed to a kernel.

static __device__ __align__(256) unsigned char scratch[kForwardScratchBytes];

hipError_t forward_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// launchers

// compute units of the current device (cached per device)
static int compute_units() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

template <int NB> struct FwdOrder;
template <> struct FwdOrder<1> { static constexpr int N = 3, S = 2; };
template <> struct FwdOrder<2> { static constexpr int N = 3, S = 4; };
template <> struct FwdOrder<4> { static constexpr int N = 3, S = 8; };

template <int NB, int DK, int DV, typename F, typename TIO>
static hipError_t run_forward_nb(const void* Q, const void* K, const void* V, const float* beta,
                                 const float* g, const float* S0, void* O, float* Sfin, void* ws,
                                 int B, int L, int H, int N, int S, int mode, float scale,
                                 int phases, hipStream_t st, const Packed& pk) {
  constexpr int DN = FwdOrder<NB>::N, DS = FwdOrder<NB>::S;
  const bool packed = pk.cu != nullptr;
  const int64_t n = packed ? (int64_t)pk.nchunks * H : (int64_t)B * H * (L / (16 * NB));
#define GDN_FWD1(SM, NC_, SC_, EX)                                                             \
  do {                                                                                         \
    if (packed)                                                                                \
      hipLaunchKernelGGL((k_fwd_chunk<NB, DK, DV, F, SM, NC_, SC_, TIO, EX, true>),            \
                         dim3((unsigned)n), dim3(64), 0, st, (const TIO*)Q, (const TIO*)K,     \
                         (const TIO*)V, beta, g, (TIO*)ws, n, L, H, N, S, pk);                 \
    else                                                                                       \
      hipLaunchKernelGGL((k_fwd_chunk<NB, DK, DV, F, SM, NC_, SC_, TIO, EX, false>),           \
                         dim3((unsigned)n), dim3(64), 0, st, (const TIO*)Q, (const TIO*)K,     \
                         (const TIO*)V, beta, g, (TIO*)ws, n, L, H, N, S, pk);                 \
  } while (0)
  if ((phases & 1) && n > 0) {
    if (mode == kInvExact) {
      GDN_FWD1(true, 0, 0, kInvExact);
    } else if (mode == kInvInt16 || mode == kInvInt8) {
      // the integer modes run the default order with dk = dv = 128
      if constexpr (DK == 128 && DV == 128) {
        if (N != DN || S != DS) return hipErrorNotSupported;
        if (mode == kInvInt16)
          GDN_FWD1(true, DN, DS, kInvInt16);
        else
          GDN_FWD1(true, DN, DS, kInvInt8);
      } else {
        return hipErrorNotSupported;
      }
    } else if (N == DN && S == DS) {
      GDN_FWD1(true, DN, DS, kInvNeumann);
    } else if (N <= 15) {
      GDN_FWD1(true, -1, -1, kInvNeumann);
    } else {
      GDN_FWD1(false, -1, -1, kInvNeumann);
    }
  }
#undef GDN_FWD1
  if (phases & 2) {
    const unsigned nwork = (unsigned)((packed ? pk.nseq : B) * H * (DV / 16));
#define GDN_FWD2(D)                                                                            \
  do {                                                                                         \
    if (packed)                                                                                \
      hipLaunchKernelGGL((k_fwd_state<NB, DK, DV, F, TIO, D, true>), dim3(nwork), dim3(256), 0, \
                         st, (const TIO*)ws, (const TIO*)Q, g, S0, (TIO*)O, Sfin, n, B, L, H,   \
                         scale, pk);                                                           \
    else                                                                                       \
      hipLaunchKernelGGL((k_fwd_state<NB, DK, DV, F, TIO, D, false>), dim3(nwork), dim3(256),  \
                         0, st, (const TIO*)ws, (const TIO*)Q, g, S0, (TIO*)O, Sfin, n, B, L,  \
                         H, scale, pk);                                                        \
  } while (0)
    if (nwork == 0) {
      // nothing to do
    } else if constexpr (sizeof(TIO) != 2) {
      GDN_FWD2(1);  // fp32 operands: twice the registers, no room for a ring
    } else if (nwork <= (unsigned)compute_units()) {
      GDN_FWD2(3);  // one workgroup per CU: the deepest ring
    } else {
      GDN_FWD2(2);  // more workgroups than CUs: a ring of two leaves room for two per CU
    }
#undef GDN_FWD2
  }
  return hipGetLastError();
}

template <typename F, typename TIO>
static hipError_t run_forward(const void* Q, const void* K, const void* V, const float* beta,
                              const float* g, const float* S0, void* O, float* Sfin, void* ws,
                              int B, int L, int H, int dk, int dv, int C, int N, int S,
                              int mode, float scale, int phases, hipStream_t st,
                              const Packed& pk) {
#define GDN_FWD_NB(NB_)                                                                      \
  GDN_DK_SWITCH(dk, GDN_DV_SWITCH(dv, {                                                      \
    return run_forward_nb<NB_, DK, DV, F, TIO>(Q, K, V, beta, g, S0, O, Sfin, ws, B, L, H, N, \
                                              S, mode, scale, phases, st, pk);               \
  }))
  switch (C) {
    case 16: GDN_FWD_NB(1) break;
    case 32: GDN_FWD_NB(2) break;
    case 64: GDN_FWD_NB(4) break;
  }
#undef GDN_FWD_NB
  return hipErrorNotSupported;
}

static hipError_t forward_dtype(const void* Q, const void* K, const void* V, const float* beta,
                                const float* g, const float* S0, void* O, float* Sfin, void* ws,
                                int B, int L, int H, int dk, int dv, int C, int N, int S,
                                int mode, float scale, int dtype, int phases, hipStream_t st,
                                const Packed& pk) {
  if (dtype == 0)
    return run_forward<f32x4, float>(Q, K, V, beta, g, S0, O, Sfin, ws, B, L, H, dk, dv, C, N, S,
                                     mode, scale, phases, st, pk);
  if (dtype == 1)
    return run_forward<bf16x4, __bf16>(Q, K, V, beta, g, S0, O, Sfin, ws, B, L, H, dk, dv, C, N,
                                       S, mode, scale, phases, st, pk);
  return hipErrorNotSupported;
}

hipError_t launch_forward(const void* Q, const void* K, const void* V, const float* beta,
                          const float* g, const float* S0, void* O, float* Sfin, void* ws, int B,
                          int L, int H, int dk, int dv, int C, int N, int S, int mode,
                          float scale, int dtype, int phases, hipStream_t st) {
  return forward_dtype(Q, K, V, beta, g, S0, O, Sfin, ws, B, L, H, dk, dv, C, N, S, mode, scale,
                       dtype, phases, st, Packed{});
}

hipError_t launch_forward_varlen(const void* Q, const void* K, const void* V, const float* beta,
                                 const float* g, const float* S0, void* O, float* Sfin, void* ws,
                                 const int* cu, const int* off, int nseq, int nchunks, int Ttok,
                                 int H, int dk, int dv, int C, int N, int S, int mode,
                                 float scale, int dtype, hipStream_t st) {
  return forward_dtype(Q, K, V, beta, g, S0, O, Sfin, ws, 1, Ttok, H, dk, dv, C, N, S, mode,
                       scale, dtype, 3, st, Packed{cu, off, nseq, nchunks});
}

}  // namespace gdn
