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
// Stage 2, k_fwd_state: one wave per (batch, head, 16 value columns).  It
// walks the chunks of its head in order with its dk x 16 slice of S in
// registers (fp32); per chunk four product groups: W S, Q S, P V_new and
// K^T V_new.
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
__host__ __device__ constexpr int pidx(int I, int p) {
  int n = 0;
  for (int i = 0; i < I; ++i) n += i / 2 + 1;
  return n + p;
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

template <int NB, int DK, int DV, typename F, bool SMALLN, int NC, int SC, typename TIO,
          bool EXACT>
__global__ __launch_bounds__(64) void k_fwd_chunk(const TIO* __restrict__ Q,
                                                  const TIO* __restrict__ K,
                                                  const TIO* __restrict__ V,
                                                  const float* __restrict__ beta,
                                                  const float* __restrict__ g,
                                                  TIO* __restrict__ ws, int64_t n_tiles, int L,
                                                  int H, int N, int S) {
  constexpr int C = 16 * NB;
  constexpr int DMAX = DK > DV ? DK : DV;
  // bf16: V, then Q, arrive in LDS by DMA while registers are busy
  constexpr bool PREF = sizeof(TIO) == 2;
  using LY = FwdLayout<NB, DK, DV>;
  __shared__ float sb[C], sg[C], sbw[C];
  __shared__ __attribute__((aligned(16))) __bf16 sx[PREF ? NB * (DMAX / 32) * 512 : 8];
  const Chunk ch(blockIdx.x, L, H, C);
  const Lane ln = lane_here();
  load_gates<C>(beta, g, ch, L, H, sb, sg);
  for (int r = ln.id; r < C; r += 64) sbw[r] = sb[r] * __expf(sg[r]);
  __syncthreads();
  TIO* wf = ws + ch.tile * LY::W;
  TIO* uf = ws + n_tiles * LY::W + ch.tile * LY::U;
  TIO* ktf = ws + n_tiles * (LY::W + LY::U) + ch.tile * LY::KT;
  TIO* pf = ws + n_tiles * (LY::W + LY::U + LY::KT) + ch.tile * LY::P;
  const int64_t ldk = (int64_t)H * DK, ldv = (int64_t)H * DV;

  Pair<F> kp[NB][DK / 32];
  load_rows<NB, DK>(kp, K + ch.row(0, L, H, DK), ldk);
  auto prefetch_v = [&]() {
    if constexpr (PREF) {
      __builtin_amdgcn_sched_barrier(0);
      prefetch_rows_lds<NB, DV>((const __bf16*)V + ch.row(0, L, H, DV), ldv, sx);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  Acc<NB> Tr;
  chunk_inverse<NB, DK, F, SMALLN, NC, SC, EXACT>(kp, sb, sg, N, S, Tr, prefetch_v);
#pragma unroll
  for (int I = 0; I < NB; ++I) Tr.a[bidx(I, I)] = band_block<false>(Tr.a[bidx(I, I)], 0, 1, C) + eye4();

  RowP<NB, F> TR;
  scale_cols(TR, Tr, sb);
  if constexpr (PREF) {
    wait_vmem();
    apply_u_fwd<NB, DV, F>(TR, LdsRows<DV>{sx, ln.id}, uf, ln);
    // Q replaces V in LDS: every read of V above has returned its data
    __builtin_amdgcn_sched_barrier(0);
    prefetch_rows_lds<NB, DK>((const __bf16*)Q + ch.row(0, L, H, DK), ldk, sx);
    __builtin_amdgcn_sched_barrier(0);
  } else {
    Pair<F> vp[NB][DV / 32];
    load_rows<NB, DV>(vp, V + ch.row(0, L, H, DV), ldv);
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
        qp[I] = load_row8<F>(Q + ch.row(I * 16 + ln.c(), L, H, DK) + 32 * q + 8 * ln.g());
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
// Two waves per (batch, head, slice): wave 1 copies the operands of the next
// chunk from the workspace (and Q, g from the inputs) into LDS by global ->
// LDS DMA while wave 0 runs the recurrence on the current chunk from LDS.
// NST = 2 stages: the copy of chunk ck + 1 overlaps the compute of chunk ck,
// one workgroup barrier per chunk; NST = 1 (fp32 at C = 64, where a stage
// would not fit twice): copy, barrier, compute, barrier.

template <int NB, int DK, int DV, typename TIO>
struct StageLayout {
  static constexpr int NQ = DK / 32;
  static constexpr int W = 0;                                   // NB * NQ slots
  static constexpr int Q = W + NB * NQ * 512;                   // NB * NQ slots
  static constexpr int KT = Q + NB * NQ * 512;                  // (DK/16) * npair slots
  static constexpr int P = KT + (DK / 16) * npair(NB) * 512;   // npp slots
  static constexpr int U = P + npp(NB) * 512;                   // NB blocks of this slice
  static constexpr int size = U + NB * 256;                     // elements of TIO
  static constexpr int bytes = size * (int)sizeof(TIO);
  static constexpr int nst = 2 * bytes + 1024 <= 150 * 1024 ? 2 : 1;
};

// wave-wide copy of `bytes` contiguous bytes (a multiple of 16) to LDS in
// runs of 1 KB, 16 bytes per lane
__device__ __forceinline__ void dma_copy(const void* src, void* dst, int bytes, int l) {
  const char* s = (const char*)src;
  char* d = (char*)dst;
  for (int o = 0; o < bytes; o += 1024)
    if (o + 16 * l < bytes)
      __builtin_amdgcn_global_load_lds((glb_void*)(s + o + 16 * l), (lds_void*)(d + o), 16, 0, 0);
}

template <int NB, int DK, int DV, typename F, typename TIO>
__global__ __launch_bounds__(128) void k_fwd_state(const TIO* __restrict__ ws,
                                                   const TIO* __restrict__ Q,
                                                   const float* __restrict__ g,
                                                   const float* __restrict__ S0,
                                                   TIO* __restrict__ O, float* __restrict__ Sfin,
                                                   int64_t n_tiles, int B, int L, int H,
                                                   float scale) {
  constexpr int C = 16 * NB, NQ = DK / 32, NM = DK / 16, NP = npair(NB), NS = DV / 16;
  using LY = FwdLayout<NB, DK, DV>;
  using SL = StageLayout<NB, DK, DV, TIO>;
  constexpr int NST = SL::nst;
  __shared__ __attribute__((aligned(16))) TIO stg[NST][SL::size];
  __shared__ __attribute__((aligned(16))) float sgam[NST][C];
  const int BH = B * H, nc = L / C;
  // work item -> (head bh = b H + h, slice j); when BH is a multiple of 8 the
  // slices of one head share an XCD (work items are dealt to the 8 XCDs in
  // turn), so the W, K^T, P and Q runs all of them read meet in one L2
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
  const int b = bh / H, h = bh - b * H;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const Lane ln = lane_here();
  const int l = ln.id;
  const int64_t ldq = (int64_t)H * DK, ldo = (int64_t)H * DV;

  if (wv == 1) {
    // ---- producer
    auto copy = [&](int ck, int st) {
      const int64_t tile = (int64_t)bh * nc + ck;
      const int64_t tok0 = (int64_t)b * L + ck * C;
      TIO* s = stg[st];
      dma_copy(ws + tile * LY::W, s + SL::W, (int)(LY::W * sizeof(TIO)), l);
      dma_copy(ws + n_tiles * LY::W + tile * LY::U + j * NB * 256, s + SL::U,
               NB * 256 * (int)sizeof(TIO), l);
      dma_copy(ws + n_tiles * (LY::W + LY::U) + tile * LY::KT, s + SL::KT,
               (int)(LY::KT * sizeof(TIO)), l);
      dma_copy(ws + n_tiles * (LY::W + LY::U + LY::KT) + tile * LY::P, s + SL::P,
               (int)(LY::P * sizeof(TIO)), l);
      // Q rows gathered into slots (I, q); fp32 as two 16-byte halves
#pragma unroll
      for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const TIO* src = Q + (tok0 + I * 16 + ln.c()) * ldq + (int64_t)h * DK + 32 * q + 8 * ln.g();
          TIO* dst = s + SL::Q + (I * NQ + q) * 512;
#pragma unroll
          for (int p = 0; p < (int)sizeof(TIO) / 2; ++p)
            __builtin_amdgcn_global_load_lds((glb_void*)(src + p * (16 / sizeof(TIO))),
                                             (lds_void*)(dst + p * 256), 16, 0, 0);
        }
      if (l < C)
        __builtin_amdgcn_global_load_lds((glb_void*)(g + (tok0 + l) * H + h),
                                         (lds_void*)sgam[st], 4, 0, 0);
    };
    if (NST == 2 && nc > 0) copy(0, 0);
    for (int ck = 0; ck < nc; ++ck) {
      if (NST == 1) copy(ck, 0);
      wait_vmem();  // chunk ck has landed
      __syncthreads();
      if (NST == 2) {
        // the stage of chunk ck - 1 is free: wave 0 has passed this barrier
        if (ck + 1 < nc) copy(ck + 1, (ck + 1) & 1);
      } else {
        __syncthreads();  // wave 0 is done with the stage
      }
    }
    return;
  }

  // ---- consumer: the recurrence
  const int gq = ln.g(), c = ln.c();
  const int jq = j >> 1, jh = j & 1;
  const int dvcol = 32 * jq + 8 * (c >> 2) + 4 * jh + (c & 3);  // column c of the slice
  const int ocol = 32 * jq + 8 * gq + 4 * jh;                   // columns 4g .. 4g + 3
  const int64_t sbase = (int64_t)bh * DK * DV;
  f32x4 st[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int dk = 32 * (m >> 1) + 8 * gq + 4 * (m & 1) + v;
      st[m][v] = S0 ? S0[sbase + (int64_t)dk * DV + dvcol] : 0.f;
    }
  // Per chunk four phases; each issues the LDS reads of the next phase's
  // operands before its own MFMAs (sched_barrier keeps the order), so the
  // reads of a phase arrive while the previous phase computes.
  for (int ck = 0; ck < nc; ++ck) {
    __syncthreads();  // chunk ck is in stage ck % NST
    const TIO* s = stg[NST == 2 ? (ck & 1) : 0];
    const float* gg = sgam[NST == 2 ? (ck & 1) : 0];
    const int64_t tok0 = (int64_t)b * L + ck * C;
    // phase 0: W and U reads; the state as MFMA operands
    Pair<F> wq[NB][NQ];
    f32x4 vn[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      vn[I] = load4(s + SL::U + I * 256 + 4 * l);
#pragma unroll
      for (int q = 0; q < NQ; ++q) wq[I][q] = slot_load<F>(s + SL::W + (I * NQ + q) * 512, l);
    }
    Pair<F> sp[NQ], nsp[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      sp[q] = Pair<F>::make(st[2 * q], st[2 * q + 1]);
      nsp[q] = Pair<F>::make(-st[2 * q], -st[2 * q + 1]);
    }
    __builtin_amdgcn_sched_barrier(0);
    // phase 1: Q reads; V_new = U - W S (column form)
    Pair<F> qq[NB][NQ];
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
      for (int q = 0; q < NQ; ++q) qq[I][q] = slot_load<F>(s + SL::Q + (I * NQ + q) * 512, l);
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int I = 0; I < NB; ++I) vn[I] = Pair<F>::template mma<false>(wq[I][q], nsp[q], vn[I]);
    __builtin_amdgcn_sched_barrier(0);
    // phase 2: K^T and P reads; O = e^gamma Q S (row form), from the state
    // entering the chunk
    Pair<F> kt[NM][NP], pp[npp(NB)];
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int p = 0; p < NP; ++p) kt[m][p] = slot_load<F>(s + SL::KT + (m * NP + p) * 512, l);
#pragma unroll
    for (int k = 0; k < npp(NB); ++k) pp[k] = slot_load<F>(s + SL::P + k * 512, l);
    const float glast = gg[C - 1];
    f32x4 o[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) o[I] = zero4();
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int I = 0; I < NB; ++I) o[I] = Pair<F>::template mma<true>(qq[I][q], sp[q], o[I]);
    __builtin_amdgcn_sched_barrier(0);
    // phase 3: V_new as operands, decayed to the chunk end for the state
    // update; O += P V_new; S = e^{gamma_last} S + K^T V_d
    Pair<F> vp[NP], vdp[NP];
    {
      f32x4 vd[NB];
#pragma unroll
      for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int v = 0; v < 4; ++v) vd[I][v] = vn[I][v] * __expf(glast - gg[I * 16 + 4 * gq + v]);
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        vp[p] = Pair<F>::make(vn[2 * p], 2 * p + 1 < NB ? vn[2 * p + 1] : zero4());
        vdp[p] = Pair<F>::make(vd[2 * p], 2 * p + 1 < NB ? vd[2 * p + 1] : zero4());
      }
    }
    const float el = __expf(glast);
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      f32x4 acc = el * st[m];
#pragma unroll
      for (int p = 0; p < NP; ++p) acc = Pair<F>::template mma<false>(kt[m][p], vdp[p], acc);
      st[m] = acc;
    }
#pragma unroll
    for (int I = 0; I < NB; ++I) {
      o[I] *= __expf(gg[I * 16 + c]);
#pragma unroll
      for (int p = 0; 2 * p <= I; ++p)
        o[I] = Pair<F>::template mma<true>(pp[pidx(I, p)], vp[p], o[I]);
      store4(O + (tok0 + I * 16 + c) * ldo + (int64_t)h * DV + ocol, scale * o[I]);
    }
    if (NST == 1) __syncthreads();  // the stage may be refilled
  }
  if (Sfin) {
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int dk = 32 * (m >> 1) + 8 * gq + 4 * (m & 1) + v;
        Sfin[sbase + (int64_t)dk * DV + dvcol] = st[m][v];
      }
  }
}

// ---------------------------------------------------------------------------
// launchers

template <int NB> struct FwdOrder;
template <> struct FwdOrder<1> { static constexpr int N = 3, S = 2; };
template <> struct FwdOrder<2> { static constexpr int N = 3, S = 4; };
template <> struct FwdOrder<4> { static constexpr int N = 3, S = 8; };

template <int NB, int DK, int DV, typename F, typename TIO>
static hipError_t run_forward_nb(const void* Q, const void* K, const void* V, const float* beta,
                                 const float* g, const float* S0, void* O, float* Sfin, void* ws,
                                 int B, int L, int H, int N, int S, bool exact, float scale,
                                 int phases, hipStream_t st) {
  constexpr int DN = FwdOrder<NB>::N, DS = FwdOrder<NB>::S;
  const int64_t n = (int64_t)B * H * (L / (16 * NB));
#define GDN_FWD1(SM, NC_, SC_, EX)                                                           \
  hipLaunchKernelGGL((k_fwd_chunk<NB, DK, DV, F, SM, NC_, SC_, TIO, EX>), dim3((unsigned)n), \
                     dim3(64), 0, st, (const TIO*)Q, (const TIO*)K, (const TIO*)V, beta, g,  \
                     (TIO*)ws, n, L, H, N, S)
  if ((phases & 1) && n > 0) {
    if (exact)
      GDN_FWD1(true, 0, 0, true);
    else if (N == DN && S == DS)
      GDN_FWD1(true, DN, DS, false);
    else if (N <= 15)
      GDN_FWD1(true, -1, -1, false);
    else
      GDN_FWD1(false, -1, -1, false);
  }
#undef GDN_FWD1
  if (phases & 2) {
    const unsigned nwork = (unsigned)(B * H * (DV / 16));
    hipLaunchKernelGGL((k_fwd_state<NB, DK, DV, F, TIO>), dim3(nwork), dim3(128), 0, st,
                       (const TIO*)ws, (const TIO*)Q, g, S0, (TIO*)O, Sfin, n, B, L, H, scale);
  }
  return hipGetLastError();
}

template <typename F, typename TIO>
static hipError_t run_forward(const void* Q, const void* K, const void* V, const float* beta,
                              const float* g, const float* S0, void* O, float* Sfin, void* ws,
                              int B, int L, int H, int dk, int dv, int C, int N, int S,
                              bool exact, float scale, int phases, hipStream_t st) {
#define GDN_FWD_NB(NB_)                                                                     \
  GDN_DK_SWITCH(dk, GDN_DV_SWITCH(dv, {                                                     \
    return run_forward_nb<NB_, DK, DV, F, TIO>(Q, K, V, beta, g, S0, O, Sfin, ws, B, L, H, N, \
                                              S, exact, scale, phases, st);                 \
  }))
  switch (C) {
    case 16: GDN_FWD_NB(1) break;
    case 32: GDN_FWD_NB(2) break;
    case 64: GDN_FWD_NB(4) break;
  }
#undef GDN_FWD_NB
  return hipErrorNotSupported;
}

hipError_t launch_forward(const void* Q, const void* K, const void* V, const float* beta,
                          const float* g, const float* S0, void* O, float* Sfin, void* ws, int B,
                          int L, int H, int dk, int dv, int C, int N, int S, bool exact,
                          float scale, int dtype, int phases, hipStream_t st) {
  if (dtype == 0)
    return run_forward<f32x4, float>(Q, K, V, beta, g, S0, O, Sfin, ws, B, L, H, dk, dv, C, N, S,
                                     exact, scale, phases, st);
  if (dtype == 1)
    return run_forward<bf16x4, __bf16>(Q, K, V, beta, g, S0, O, Sfin, ws, B, L, H, dk, dv, C, N,
                                       S, exact, scale, phases, st);
  return hipErrorNotSupported;
}

}  // namespace gdn
