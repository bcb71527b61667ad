// api.cpp -- the extern "C" boundary declared in include/gdninv.h.
// Validates every argument before anything is enqueued, then dispatches to
// the launchers.  Holds no state.
#include "gdninv.h"

#include <stdint.h>

#include "launch.hpp"

namespace {

// A 1-D launch of n workgroups of `block` work items fits HIP's grid when
// n <= 2^31 - 1 and n * block <= 2^32 - 1.  Every launch here is one
// workgroup per tile (or per (head, slice) of the state pass), of 64 work
// items, 128 for the two-wave C = 128 kernels (fused path and integer
// inverse) and 256 for the C = 128 quantiser and the state pass; the fused
// kernels that put 2 or 4 tiles in one workgroup launch as many work items
// per tile in fewer workgroups, so the per-tile check covers them.
bool grid_ok(int64_t n, int block) {
  return n >= 0 && n <= 0x7fffffffLL && n * block <= 0xffffffffLL;
}
int two_wave(int C) { return C == 128 ? 128 : 64; }

bool valid_C(int C) { return C == 16 || C == 32 || C == 64 || C == 128; }
bool valid_d(int d) { return d == 64 || d == 128; }
bool fdtype(int t) { return t == GDN_F32 || t == GDN_BF16; }
int64_t esize(int t) { return t == GDN_F32 ? 4 : (t == GDN_BF16 ? 2 : 1); }
bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// [p, p + bytes) and [q, q + qbytes) intersect
bool overlap(const void* p, int64_t bytes, const void* q, int64_t qbytes) {
  if (!p || !q || bytes <= 0 || qbytes <= 0) return false;
  const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
  return a < b + (uintptr_t)qbytes && b < a + (uintptr_t)bytes;
}

// exponents per tile of the integer paths: C = 128 runs three blocks
int64_t nexp(int C) { return C == 128 ? 3 : 1; }

// The inverse modes of the layer forward: 0 T_hat(N, S), 1 exact, 2 T_hat(N, S)
// on 16-bit codes, 3 on 8-bit codes.  The integer modes run the default order
// with dk = dv = 128 (anything else: GDN_ERR_UNSUPPORTED).
int forward_mode_check(int mode, int C, int N, int S, int dk, int dv, bool prep) {
  if (mode < 0 || mode > 3) return GDN_ERR_PARAM;
  if (prep && mode != 1) {
    const int lim = (C == 128 ? 64 : C) - 1;
    if (N < 0 || S < 0 || N > lim || S > lim) return GDN_ERR_PARAM;
  }
  if (prep && mode >= 2) {
    const int dn = 3, ds = C == 16 ? 2 : C == 32 ? 4 : 8;
    if (N != dn || S != ds || dk != 128 || dv != 128) return GDN_ERR_UNSUPPORTED;
  }
  return GDN_OK;
}

int order_ok(int C, int N, int S) {
  const int lim = (C == 128 ? 64 : C) - 1;  // C = 128 runs 64-blocks
  return N >= 0 && S >= 0 && N <= lim && S <= lim;
}

int hip_status(hipError_t e) {
  if (e == hipSuccess) return GDN_OK;
  if (e == hipErrorNotSupported) return GDN_ERR_UNSUPPORTED;
  return GDN_ERR_HIP;
}

// common checks of the [B, L, H, d] entry points (one workgroup of `block`
// work items per tile); fills the tile count
int check_chunked(int B, int L, int H, int C, int64_t* n_tiles, int block) {
  if (B < 0 || L < 0 || H < 0 || !valid_C(C) || L % C != 0) return GDN_ERR_SHAPE;
  const int64_t n = (int64_t)B * H * (L / C);
  if (!grid_ok(n, block)) return GDN_ERR_SHAPE;
  *n_tiles = n;
  return GDN_OK;
}

}  // namespace

extern "C" {

int gdn_abi_version(void) { return GDN_ABI_VERSION; }

const char* gdn_status_string(int status) {
  switch (status) {
    case GDN_OK: return "ok";
    case GDN_ERR_NULL: return "a required pointer is NULL";
    case GDN_ERR_SHAPE: return "size out of range (C in {16,32,64,128}, L % C == 0, d in {64,128})";
    case GDN_ERR_PARAM: return "order out of range (0 <= N, S <= C - 1; 63 for C = 128)";
    case GDN_ERR_DTYPE: return "unsupported dtype";
    case GDN_ERR_ALIGN: return "pointer not 16-byte aligned";
    case GDN_ERR_ALIAS: return "an output overlaps an input";
    case GDN_ERR_HIP: return "HIP runtime error at launch";
    case GDN_ERR_UNSUPPORTED: return "combination not implemented by the library";
    case GDN_ERR_WORKSPACE: return "workspace smaller than gdn_chunk_forward_workspace()";
  }
  return "unknown status";
}

int gdn_default_order(int C, int* N, int* S) {
  if (!N || !S) return GDN_ERR_NULL;
  switch (C) {
    case 16: *N = 3; *S = 2; return GDN_OK;
    case 32: *N = 3; *S = 4; return GDN_OK;
    case 64: *N = 3; *S = 8; return GDN_OK;
    case 128: *N = 3; *S = 8; return GDN_OK;
  }
  return GDN_ERR_SHAPE;
}

int gdn_build_A(const void* K, const float* beta, const float* g, void* A, int B, int L, int H,
                int dk, int C, int k_dtype, int a_dtype, void* stream) {
  int64_t n = 0;
  if (int r = check_chunked(B, L, H, C, &n, 64)) return r;
  if (!valid_d(dk)) return GDN_ERR_SHAPE;
  if (!fdtype(k_dtype) || !fdtype(a_dtype)) return GDN_ERR_DTYPE;
  if (n == 0) return GDN_OK;
  if (!K || !beta || !g || !A) return GDN_ERR_NULL;
  if (!aligned(K) || !aligned(beta) || !aligned(g) || !aligned(A)) return GDN_ERR_ALIGN;
  const int64_t tok = (int64_t)B * L * H;
  const int64_t a_bytes = n * C * C * esize(a_dtype);
  if (overlap(A, a_bytes, K, tok * dk * esize(k_dtype)) || overlap(A, a_bytes, beta, tok * 4) ||
      overlap(A, a_bytes, g, tok * 4))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_build_A(K, beta, g, A, B, L, H, dk, C, k_dtype, a_dtype,
                                        (hipStream_t)stream));
}

int gdn_chunk_inverse_neumann(const void* A, void* Tinv, int64_t n_tiles, int C, int N, int S,
                              int dtype, void* stream) {
  if (!valid_C(C) || !grid_ok(n_tiles, 64)) return GDN_ERR_SHAPE;
  if (!order_ok(C, N, S)) return GDN_ERR_PARAM;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (n_tiles == 0) return GDN_OK;
  if (!A || !Tinv) return GDN_ERR_NULL;
  if (!aligned(A) || !aligned(Tinv)) return GDN_ERR_ALIGN;
  const int64_t bytes = n_tiles * C * C * esize(dtype);
  if (overlap(A, bytes, Tinv, bytes)) return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_neumann(A, Tinv, n_tiles, C, N, S, dtype, (hipStream_t)stream));
}

int gdn_chunk_inverse_fwdsub(const void* A, void* Tinv, int64_t n_tiles, int C, int dtype,
                             void* stream) {
  if (!valid_C(C) || !grid_ok(n_tiles, 64)) return GDN_ERR_SHAPE;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (n_tiles == 0) return GDN_OK;
  if (!A || !Tinv) return GDN_ERR_NULL;
  if (!aligned(A) || !aligned(Tinv)) return GDN_ERR_ALIGN;
  const int64_t bytes = n_tiles * C * C * esize(dtype);
  if (overlap(A, bytes, Tinv, bytes)) return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_fwdsub(A, Tinv, n_tiles, C, dtype, (hipStream_t)stream));
}

int gdn_chunk_inverse_blockwise(const void* A, void* Tinv, int64_t n_tiles, int C, int dtype,
                                void* stream) {
  if (!valid_C(C) || !grid_ok(n_tiles, 64)) return GDN_ERR_SHAPE;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (n_tiles == 0) return GDN_OK;
  if (!A || !Tinv) return GDN_ERR_NULL;
  if (!aligned(A) || !aligned(Tinv)) return GDN_ERR_ALIGN;
  const int64_t bytes = n_tiles * C * C * esize(dtype);
  if (overlap(A, bytes, Tinv, bytes)) return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_blockwise(A, Tinv, n_tiles, C, dtype, (hipStream_t)stream));
}

int gdn_wy_apply(const void* Tinv, const void* K, const void* V, const float* beta, void* W,
                 void* U, int B, int L, int H, int dk, int dv, int C, int dtype, void* stream) {
  int64_t n = 0;
  if (int r = check_chunked(B, L, H, C, &n, 64)) return r;
  if (!valid_d(dk) || !valid_d(dv)) return GDN_ERR_SHAPE;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (n == 0) return GDN_OK;
  if (!Tinv || !K || !V || !beta || !W || !U) return GDN_ERR_NULL;
  if (!aligned(Tinv) || !aligned(K) || !aligned(V) || !aligned(beta) || !aligned(W) ||
      !aligned(U))
    return GDN_ERR_ALIGN;
  const int64_t tok = (int64_t)B * L * H, es = esize(dtype);
  const int64_t tb = n * C * C * es, kb = tok * dk * es, vb = tok * dv * es, bb = tok * 4;
  const void* ins[4] = {Tinv, K, V, beta};
  const int64_t inb[4] = {tb, kb, vb, bb};
  for (int i = 0; i < 4; ++i)
    if (overlap(W, kb, ins[i], inb[i]) || overlap(U, vb, ins[i], inb[i])) return GDN_ERR_ALIAS;
  if (overlap(W, kb, U, vb)) return GDN_ERR_ALIAS;
  return hip_status(
      gdn::launch_wy(Tinv, K, V, beta, W, U, B, L, H, dk, dv, C, dtype, (hipStream_t)stream));
}

namespace {
int wy_fused(const void* K, const void* V, const float* beta, const float* g, void* W, void* U,
             void* Tinv, int B, int L, int H, int dk, int dv, int C, int N, int S, int dtype,
             bool exact, void* stream) {
  int64_t n = 0;
  if (int r = check_chunked(B, L, H, C, &n, two_wave(C))) return r;
  if (!valid_d(dk) || !valid_d(dv)) return GDN_ERR_SHAPE;
  if (!exact && !order_ok(C, N, S)) return GDN_ERR_PARAM;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (n == 0) return GDN_OK;
  if (!K || !V || !beta || !g || !W || !U) return GDN_ERR_NULL;
  if (!aligned(K) || !aligned(V) || !aligned(beta) || !aligned(g) || !aligned(W) ||
      !aligned(U) || (Tinv && !aligned(Tinv)))
    return GDN_ERR_ALIGN;
  const int64_t tok = (int64_t)B * L * H, es = esize(dtype);
  const int64_t kb = tok * dk * es, vb = tok * dv * es, bb = tok * 4, tb = n * C * C * es;
  const void* ins[4] = {K, V, beta, g};
  const int64_t inb[4] = {kb, vb, bb, bb};
  for (int i = 0; i < 4; ++i)
    if (overlap(W, kb, ins[i], inb[i]) || overlap(U, vb, ins[i], inb[i]) ||
        overlap(Tinv, tb, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(W, kb, U, vb) || overlap(W, kb, Tinv, tb) || overlap(U, vb, Tinv, tb))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_fused(K, V, beta, g, W, U, Tinv, B, L, H, dk, dv, C, N, S, dtype,
                                      exact, (hipStream_t)stream));
}
}  // namespace

int gdn_chunk_wy_fused(const void* K, const void* V, const float* beta, const float* g, void* W,
                       void* U, void* Tinv, int B, int L, int H, int dk, int dv, int C, int N,
                       int S, int dtype, void* stream) {
  return wy_fused(K, V, beta, g, W, U, Tinv, B, L, H, dk, dv, C, N, S, dtype, false, stream);
}

int gdn_chunk_wy_fused_blockwise(const void* K, const void* V, const float* beta, const float* g,
                                 void* W, void* U, void* Tinv, int B, int L, int H, int dk, int dv,
                                 int C, int dtype, void* stream) {
  return wy_fused(K, V, beta, g, W, U, Tinv, B, L, H, dk, dv, C, 0, 0, dtype, true, stream);
}

int gdn_chunk_wy_fused_varlen(const void* K, const void* V, const float* beta, const float* g,
                              void* W, void* U, void* Tinv, const int32_t* cu_seqlens,
                              const int32_t* chunk_offsets, int nseq, int n_chunks, int T, int H,
                              int dk, int dv, int C, int N, int S, int exact, int dtype,
                              void* stream) {
  if (T < 0 || H < 0 || nseq < 0 || n_chunks < 0) return GDN_ERR_SHAPE;
  if (!valid_C(C) || !valid_d(dk) || !valid_d(dv)) return GDN_ERR_SHAPE;
  if (nseq == 0 && n_chunks != 0) return GDN_ERR_SHAPE;
  if (n_chunks > T || !grid_ok((int64_t)n_chunks * H, two_wave(C))) return GDN_ERR_SHAPE;
  if (exact != 0 && exact != 1) return GDN_ERR_PARAM;
  if (!exact && !order_ok(C, N, S)) return GDN_ERR_PARAM;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (n_chunks == 0 || H == 0) return GDN_OK;
  if (!K || !V || !beta || !g || !W || !U || !cu_seqlens || !chunk_offsets) return GDN_ERR_NULL;
  if (!aligned(K) || !aligned(V) || !aligned(beta) || !aligned(g) || !aligned(W) ||
      !aligned(U) || (Tinv && !aligned(Tinv)) || (reinterpret_cast<uintptr_t>(cu_seqlens) & 3) ||
      (reinterpret_cast<uintptr_t>(chunk_offsets) & 3))
    return GDN_ERR_ALIGN;
  const int64_t tok = (int64_t)T * H, es = esize(dtype);
  const int64_t kb = tok * dk * es, vb = tok * dv * es, bb = tok * 4;
  const int64_t tb = (int64_t)H * n_chunks * C * C * es, qb = ((int64_t)nseq + 1) * 4;
  const void* ins[6] = {K, V, beta, g, cu_seqlens, chunk_offsets};
  const int64_t inb[6] = {kb, vb, bb, bb, qb, qb};
  for (int i = 0; i < 6; ++i)
    if (overlap(W, kb, ins[i], inb[i]) || overlap(U, vb, ins[i], inb[i]) ||
        overlap(Tinv, tb, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(W, kb, U, vb) || overlap(W, kb, Tinv, tb) || overlap(U, vb, Tinv, tb))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_fused_varlen(K, V, beta, g, W, U, Tinv, cu_seqlens, chunk_offsets,
                                             nseq, n_chunks, T, H, dk, dv, C, N, S, dtype,
                                             exact != 0, (hipStream_t)stream));
}

int gdn_chunk_forward_varlen(const void* Q, const void* K, const void* V, const float* beta,
                             const float* g, const float* S0, void* O, float* S_final,
                             void* workspace, int64_t workspace_bytes,
                             const int32_t* cu_seqlens, const int32_t* chunk_offsets, int nseq,
                             int n_chunks, int T, int H, int dk, int dv, int C, int N, int S,
                             int exact, float scale, int dtype, void* stream) {
  if (T < 0 || H < 0 || nseq < 0 || n_chunks < 0) return GDN_ERR_SHAPE;
  if (!valid_C(C) || !valid_d(dk) || !valid_d(dv)) return GDN_ERR_SHAPE;
  if (nseq == 0 && n_chunks != 0) return GDN_ERR_SHAPE;
  if (n_chunks > T || !grid_ok((int64_t)n_chunks * H, 64)) return GDN_ERR_SHAPE;
  if (!grid_ok((int64_t)nseq * H * (dv / 16), 256)) return GDN_ERR_SHAPE;
  if (int r = forward_mode_check(exact, C, N, S, dk, dv, true)) return r;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (C == 128) return GDN_ERR_UNSUPPORTED;
  if (nseq == 0 || H == 0) return GDN_OK;
  const int64_t es = esize(dtype), tok = (int64_t)T * H;
  const int64_t n = (int64_t)n_chunks * H;
  const int64_t need = n * gdn::fwd_workspace_elems(C, dk, dv) * es;
  if (!cu_seqlens || !chunk_offsets) return GDN_ERR_NULL;
  if (n > 0) {
    if (!Q || !K || !V || !beta || !g || !O || !workspace) return GDN_ERR_NULL;
    if (workspace_bytes < need) return GDN_ERR_WORKSPACE;
  } else {
    Q = K = V = nullptr, beta = g = nullptr, O = nullptr, workspace = nullptr;
  }
  const void* ptrs[9] = {Q, K, V, beta, g, S0, O, S_final, workspace};
  for (const void* p : ptrs)
    if (p && !aligned(p)) return GDN_ERR_ALIGN;
  if ((reinterpret_cast<uintptr_t>(cu_seqlens) & 3) ||
      (reinterpret_cast<uintptr_t>(chunk_offsets) & 3))
    return GDN_ERR_ALIGN;
  const int64_t qb = tok * dk * es, vb = tok * dv * es, bb = tok * 4;
  const int64_t sb = (int64_t)nseq * H * dk * dv * 4, tb = ((int64_t)nseq + 1) * 4;
  const void* ins[8] = {Q, K, V, beta, g, S0, cu_seqlens, chunk_offsets};
  const int64_t inb[8] = {qb, qb, vb, bb, bb, sb, tb, tb};
  const void* outs[3] = {O, workspace, S_final};
  const int64_t outb[3] = {vb, need, sb};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 8; ++i) {
      if (o == 2 && i == 5 && S_final == S0) continue;  // in-place state update
      if (overlap(outs[o], outb[o], ins[i], inb[i])) return GDN_ERR_ALIAS;
    }
    for (int o2 = o + 1; o2 < 3; ++o2)
      if (overlap(outs[o], outb[o], outs[o2], outb[o2])) return GDN_ERR_ALIAS;
  }
  return hip_status(gdn::launch_forward_varlen(Q, K, V, beta, g, S0, O, S_final, workspace,
                                               cu_seqlens, chunk_offsets, nseq, n_chunks, T, H,
                                               dk, dv, C, N, S, exact, scale, dtype,
                                               (hipStream_t)stream));
}

int gdn_quantize_tiles_i8(const float* A, int8_t* Aq, int32_t* eA, int64_t n_tiles, int C,
                          void* stream) {
  if (!valid_C(C) || !grid_ok(n_tiles, C == 128 ? 256 : 64))
    return GDN_ERR_SHAPE;
  if (n_tiles == 0) return GDN_OK;
  if (!A || !Aq || !eA) return GDN_ERR_NULL;
  if (!aligned(A) || !aligned(Aq) || !aligned(eA)) return GDN_ERR_ALIGN;
  const int64_t ab = n_tiles * C * C * 4, qb = n_tiles * C * C, eb = n_tiles * 4 * nexp(C);
  if (overlap(Aq, qb, A, ab) || overlap(eA, eb, A, ab) || overlap(Aq, qb, eA, eb))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_quantize_i8(A, Aq, eA, n_tiles, C, (hipStream_t)stream));
}

int gdn_chunk_inverse_neumann_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                                 float* Tdeq, int64_t n_tiles, int C, int N, int S, int flags,
                                 void* stream) {
  if (!valid_C(C) || !grid_ok(n_tiles, two_wave(C)))
    return GDN_ERR_SHAPE;
  if (!order_ok(C, N, S) || (flags & ~GDN_INT_PLAIN)) return GDN_ERR_PARAM;
  if ((flags & GDN_INT_PLAIN) && C == 128) return GDN_ERR_UNSUPPORTED;
  if (n_tiles == 0) return GDN_OK;
  if (!Aq || !eA || !Tq || !eT) return GDN_ERR_NULL;
  if (!aligned(Aq) || !aligned(eA) || !aligned(Tq) || !aligned(eT) || (Tdeq && !aligned(Tdeq)))
    return GDN_ERR_ALIGN;
  const int64_t qb = n_tiles * C * C, eb = n_tiles * 4 * nexp(C), db = n_tiles * C * C * 4;
  const void* ins[2] = {Aq, eA};
  const int64_t inb[2] = {qb, eb};
  for (int i = 0; i < 2; ++i)
    if (overlap(Tq, qb, ins[i], inb[i]) || overlap(eT, eb, ins[i], inb[i]) ||
        overlap(Tdeq, db, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(Tq, qb, eT, eb) || overlap(Tq, qb, Tdeq, db) || overlap(eT, eb, Tdeq, db))
    return GDN_ERR_ALIAS;
  return hip_status(
      gdn::launch_neumann_i8(Aq, eA, Tq, eT, Tdeq, n_tiles, C, N, S, (flags & GDN_INT_PLAIN) != 0,
                             (hipStream_t)stream));
}

int gdn_chunk_inverse_neumann_i8_fused(const void* K, const float* beta, const float* g,
                                       int8_t* Tq, int32_t* eT, float* Tdeq, int B, int L, int H,
                                       int dk, int C, int N, int S, int k_dtype, void* stream) {
  int64_t n = 0;
  if (int r = check_chunked(B, L, H, C, &n, two_wave(C))) return r;
  if (!valid_d(dk)) return GDN_ERR_SHAPE;
  if (!order_ok(C, N, S)) return GDN_ERR_PARAM;
  if (!fdtype(k_dtype)) return GDN_ERR_DTYPE;
  if (n == 0) return GDN_OK;
  if (!K || !beta || !g || !Tq || !eT) return GDN_ERR_NULL;
  if (!aligned(K) || !aligned(beta) || !aligned(g) || !aligned(Tq) || !aligned(eT) ||
      (Tdeq && !aligned(Tdeq)))
    return GDN_ERR_ALIGN;
  const int64_t tok = (int64_t)B * L * H;
  const int64_t qb = n * C * C, eb = n * 4 * nexp(C), db = n * C * C * 4;
  const void* ins[3] = {K, beta, g};
  const int64_t inb[3] = {tok * dk * esize(k_dtype), tok * 4, tok * 4};
  for (int i = 0; i < 3; ++i)
    if (overlap(Tq, qb, ins[i], inb[i]) || overlap(eT, eb, ins[i], inb[i]) ||
        overlap(Tdeq, db, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(Tq, qb, eT, eb) || overlap(Tq, qb, Tdeq, db) || overlap(eT, eb, Tdeq, db))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_inverse_i8_fused(K, beta, g, Tq, eT, Tdeq, B, L, H, dk, C, N, S,
                                                 k_dtype, (hipStream_t)stream));
}

int gdn_quantize_tiles_i16(const float* A, int16_t* Aq, int32_t* eA, int64_t n_tiles, int C,
                           void* stream) {
  if (!valid_C(C) || !grid_ok(n_tiles, C == 128 ? 256 : 64))
    return GDN_ERR_SHAPE;
  if (n_tiles == 0) return GDN_OK;
  if (!A || !Aq || !eA) return GDN_ERR_NULL;
  if (!aligned(A) || !aligned(Aq) || !aligned(eA)) return GDN_ERR_ALIGN;
  const int64_t ab = n_tiles * C * C * 4, qb = n_tiles * C * C * 2, eb = n_tiles * 4 * nexp(C);
  if (overlap(Aq, qb, A, ab) || overlap(eA, eb, A, ab) || overlap(Aq, qb, eA, eb))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_quantize_i16(A, Aq, eA, n_tiles, C, (hipStream_t)stream));
}

int gdn_chunk_inverse_neumann_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq,
                                  int32_t* eT, float* Tdeq, int64_t n_tiles, int C, int N, int S,
                                  int flags, void* stream) {
  if (!valid_C(C) || !grid_ok(n_tiles, two_wave(C)))
    return GDN_ERR_SHAPE;
  if (!order_ok(C, N, S) || (flags & ~GDN_INT_PLAIN)) return GDN_ERR_PARAM;
  if ((flags & GDN_INT_PLAIN) && C == 128) return GDN_ERR_UNSUPPORTED;
  if (n_tiles == 0) return GDN_OK;
  if (!Aq || !eA || !Tq || !eT) return GDN_ERR_NULL;
  if (!aligned(Aq) || !aligned(eA) || !aligned(Tq) || !aligned(eT) || (Tdeq && !aligned(Tdeq)))
    return GDN_ERR_ALIGN;
  const int64_t qb = n_tiles * C * C * 2, eb = n_tiles * 4 * nexp(C), db = n_tiles * C * C * 4;
  const void* ins[2] = {Aq, eA};
  const int64_t inb[2] = {qb, eb};
  for (int i = 0; i < 2; ++i)
    if (overlap(Tq, qb, ins[i], inb[i]) || overlap(eT, eb, ins[i], inb[i]) ||
        overlap(Tdeq, db, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(Tq, qb, eT, eb) || overlap(Tq, qb, Tdeq, db) || overlap(eT, eb, Tdeq, db))
    return GDN_ERR_ALIAS;
  return hip_status(
      gdn::launch_neumann_i16(Aq, eA, Tq, eT, Tdeq, n_tiles, C, N, S,
                              (flags & GDN_INT_PLAIN) != 0, (hipStream_t)stream));
}

int gdn_chunk_inverse_fwdsub_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq, int32_t* eT,
                                 float* Tdeq, int64_t n_tiles, int C, void* stream) {
  if (!(C == 16 || C == 32 || C == 64) || !grid_ok(n_tiles, 64))
    return GDN_ERR_SHAPE;
  if (n_tiles == 0) return GDN_OK;
  if (!Aq || !eA || !Tq || !eT) return GDN_ERR_NULL;
  if (!aligned(Aq) || !aligned(eA) || !aligned(Tq) || !aligned(eT) || (Tdeq && !aligned(Tdeq)))
    return GDN_ERR_ALIGN;
  const int64_t qb = n_tiles * C * C * 2, eb = n_tiles * 4, db = n_tiles * C * C * 4;
  const void* ins[2] = {Aq, eA};
  const int64_t inb[2] = {qb, eb};
  for (int i = 0; i < 2; ++i)
    if (overlap(Tq, qb, ins[i], inb[i]) || overlap(eT, eb, ins[i], inb[i]) ||
        overlap(Tdeq, db, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(Tq, qb, eT, eb) || overlap(Tq, qb, Tdeq, db) || overlap(eT, eb, Tdeq, db))
    return GDN_ERR_ALIAS;
  return hip_status(
      gdn::launch_fwdsub_i16(Aq, eA, Tq, eT, Tdeq, n_tiles, C, (hipStream_t)stream));
}

int gdn_chunk_inverse_fwdsub_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                                float* Tdeq, int64_t n_tiles, int C, void* stream) {
  if (!(C == 16 || C == 32 || C == 64) || !grid_ok(n_tiles, 64))
    return GDN_ERR_SHAPE;
  if (n_tiles == 0) return GDN_OK;
  if (!Aq || !eA || !Tq || !eT) return GDN_ERR_NULL;
  if (!aligned(Aq) || !aligned(eA) || !aligned(Tq) || !aligned(eT) || (Tdeq && !aligned(Tdeq)))
    return GDN_ERR_ALIGN;
  const int64_t qb = n_tiles * C * C, eb = n_tiles * 4, db = n_tiles * C * C * 4;
  const void* ins[2] = {Aq, eA};
  const int64_t inb[2] = {qb, eb};
  for (int i = 0; i < 2; ++i)
    if (overlap(Tq, qb, ins[i], inb[i]) || overlap(eT, eb, ins[i], inb[i]) ||
        overlap(Tdeq, db, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(Tq, qb, eT, eb) || overlap(Tq, qb, Tdeq, db) || overlap(eT, eb, Tdeq, db))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_fwdsub_i8(Aq, eA, Tq, eT, Tdeq, n_tiles, C, (hipStream_t)stream));
}

int gdn_chunk_inverse_neumann_i16_fused(const void* K, const float* beta, const float* g,
                                        int16_t* Tq, int32_t* eT, float* Tdeq, int B, int L,
                                        int H, int dk, int C, int N, int S, int k_dtype,
                                        void* stream) {
  int64_t n = 0;
  if (int r = check_chunked(B, L, H, C, &n, two_wave(C))) return r;
  if (!valid_d(dk)) return GDN_ERR_SHAPE;
  if (!order_ok(C, N, S)) return GDN_ERR_PARAM;
  if (!fdtype(k_dtype)) return GDN_ERR_DTYPE;
  if (n == 0) return GDN_OK;
  if (!K || !beta || !g || !Tq || !eT) return GDN_ERR_NULL;
  if (!aligned(K) || !aligned(beta) || !aligned(g) || !aligned(Tq) || !aligned(eT) ||
      (Tdeq && !aligned(Tdeq)))
    return GDN_ERR_ALIGN;
  const int64_t tok = (int64_t)B * L * H;
  const int64_t qb = n * C * C * 2, eb = n * 4 * nexp(C), db = n * C * C * 4;
  const void* ins[3] = {K, beta, g};
  const int64_t inb[3] = {tok * dk * esize(k_dtype), tok * 4, tok * 4};
  for (int i = 0; i < 3; ++i)
    if (overlap(Tq, qb, ins[i], inb[i]) || overlap(eT, eb, ins[i], inb[i]) ||
        overlap(Tdeq, db, ins[i], inb[i]))
      return GDN_ERR_ALIAS;
  if (overlap(Tq, qb, eT, eb) || overlap(Tq, qb, Tdeq, db) || overlap(eT, eb, Tdeq, db))
    return GDN_ERR_ALIAS;
  return hip_status(gdn::launch_inverse_i16_fused(K, beta, g, Tq, eT, Tdeq, B, L, H, dk, C, N,
                                                  S, k_dtype, (hipStream_t)stream));
}

int gdn_chunk_forward_workspace(int B, int L, int H, int dk, int dv, int C, int dtype,
                                int64_t* bytes) {
  if (!bytes) return GDN_ERR_NULL;
  int64_t n = 0;
  if (int r = check_chunked(B, L, H, C, &n, 64)) return r;
  if (!valid_d(dk) || !valid_d(dv)) return GDN_ERR_SHAPE;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (C == 128) return GDN_ERR_UNSUPPORTED;
  *bytes = n * gdn::fwd_workspace_elems(C, dk, dv) * esize(dtype);
  return GDN_OK;
}

namespace {
// phases: 1 = per-chunk launch only, 2 = state pass only, 3 = both
int forward(const void* Q, const void* K, const void* V, const float* beta, const float* g,
            const float* S0, void* O, float* S_final, void* workspace, int64_t workspace_bytes,
            int B, int L, int H, int dk, int dv, int C, int N, int S, int exact, float scale,
            int dtype, int phases, void* stream) {
  int64_t n = 0;
  if (int r = check_chunked(B, L, H, C, &n, 64)) return r;
  if (!valid_d(dk) || !valid_d(dv)) return GDN_ERR_SHAPE;
  if (int r = forward_mode_check(exact, C, N, S, dk, dv, phases & 1)) return r;
  if (!fdtype(dtype)) return GDN_ERR_DTYPE;
  if (C == 128) return GDN_ERR_UNSUPPORTED;
  if (!grid_ok((int64_t)B * H * (dv / 16), 256)) return GDN_ERR_SHAPE;
  if ((int64_t)B * H == 0) return GDN_OK;
  const bool prep = phases & 1, state = phases & 2;
  const int64_t es = esize(dtype), tok = (int64_t)B * L * H;
  const int64_t need = n * gdn::fwd_workspace_elems(C, dk, dv) * es;
  if (n > 0) {
    if (!Q || !g || !workspace) return GDN_ERR_NULL;
    if (prep && (!K || !V || !beta)) return GDN_ERR_NULL;
    if (state && !O) return GDN_ERR_NULL;
    if (workspace_bytes < need) return GDN_ERR_WORKSPACE;
  } else if (!state) {
    return GDN_OK;  // no chunk to prepare
  }
  if (!prep) K = V = nullptr, beta = nullptr;
  if (!state) S0 = nullptr, O = nullptr, S_final = nullptr;
  if (n == 0) workspace = nullptr, Q = nullptr, g = nullptr, O = nullptr;
  const void* ptrs[9] = {Q, K, V, beta, g, S0, O, S_final, workspace};
  for (const void* p : ptrs)
    if (p && !aligned(p)) return GDN_ERR_ALIGN;
  const int64_t qb = tok * dk * es, vb = tok * dv * es, bb = tok * 4;
  const int64_t sb = (int64_t)B * H * dk * dv * 4;
  // every input against every output, and the outputs against each other;
  // the workspace is an output of the per-chunk launch and an input of the
  // state pass, and overlaps neither side
  const void* ins[6] = {Q, K, V, beta, g, S0};
  const int64_t inb[6] = {qb, qb, vb, bb, bb, sb};
  const void* outs[3] = {O, workspace, S_final};
  const int64_t outb[3] = {vb, need, sb};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 6; ++i) {
      if (o == 2 && i == 5 && S_final == S0) continue;  // in-place state update
      if (overlap(outs[o], outb[o], ins[i], inb[i])) return GDN_ERR_ALIAS;
    }
    for (int o2 = o + 1; o2 < 3; ++o2)
      if (overlap(outs[o], outb[o], outs[o2], outb[o2])) return GDN_ERR_ALIAS;
  }
  return hip_status(gdn::launch_forward(Q, K, V, beta, g, S0, O, S_final, workspace, B, L, H, dk,
                                        dv, C, N, S, exact, scale, dtype, phases,
                                        (hipStream_t)stream));
}
}  // namespace

int gdn_chunk_forward(const void* Q, const void* K, const void* V, const float* beta,
                      const float* g, const float* S0, void* O, float* S_final, void* workspace,
                      int64_t workspace_bytes, int B, int L, int H, int dk, int dv, int C, int N,
                      int S, int exact, float scale, int dtype, void* stream) {
  return forward(Q, K, V, beta, g, S0, O, S_final, workspace, workspace_bytes, B, L, H, dk, dv,
                 C, N, S, exact, scale, dtype, 3, stream);
}

int gdn_chunk_forward_noalloc(const void* Q, const void* K, const void* V, const float* beta,
                              const float* g, const float* S0, void* O, float* S_final, int B,
                              int L, int H, int dk, int dv, int C, int N, int S, int exact,
                              float scale, int dtype, void* stream) {
  static_assert(gdn::kForwardScratchBytes == GDN_FORWARD_SCRATCH_BYTES, "scratch size");
  // sizes first: a call that cannot fit the scratch fails before any HIP call
  int64_t need = 0;
  if (int r = gdn_chunk_forward_workspace(B, L, H, dk, dv, C, dtype, &need)) return r;
  if (need > gdn::kForwardScratchBytes) return GDN_ERR_WORKSPACE;
  void* ws = nullptr;
  if (need > 0) {
    if (gdn::forward_scratch(&ws) != hipSuccess) return GDN_ERR_HIP;
  }
  return forward(Q, K, V, beta, g, S0, O, S_final, ws, gdn::kForwardScratchBytes, B, L, H, dk,
                 dv, C, N, S, exact, scale, dtype, 3, stream);
}

int gdn_chunk_forward_prepare(const void* Q, const void* K, const void* V, const float* beta,
                              const float* g, void* workspace, int64_t workspace_bytes, int B,
                              int L, int H, int dk, int dv, int C, int N, int S, int exact,
                              int dtype, void* stream) {
  return forward(Q, K, V, beta, g, nullptr, nullptr, nullptr, workspace, workspace_bytes, B, L,
                 H, dk, dv, C, N, S, exact, 1.f, dtype, 1, stream);
}

int gdn_chunk_forward_state(const void* Q, const float* g, const float* S0, void* O,
                            float* S_final, const void* workspace, int64_t workspace_bytes, int B,
                            int L, int H, int dk, int dv, int C, float scale, int dtype,
                            void* stream) {
  return forward(Q, nullptr, nullptr, nullptr, g, S0, O, S_final, const_cast<void*>(workspace),
                 workspace_bytes, B, L, H, dk, dv, C, 0, 0, 0, scale, dtype, 2, stream);
}

}  // extern "C"
