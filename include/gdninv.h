/*
 * gdninv.h -- C ABI of the MI355X (gfx950) chunk-inverse library for
 * chunk-wise Gated DeltaNet.
 *
 * Problem (arXiv 2606.06034, Section 2.1): for every (batch, head, chunk)
 * tile, invert the unit lower-triangular C x C matrix (I + A), where
 *     A_ij = beta_i (k_i . k_j) exp(g_i - g_j)   for i > j,   else 0,
 * and apply the inverse to the chunk's keys and values.  The paper writes
 * the inverse as (I - A)^-1; this library uses the Gated DeltaNet sign, so
 * every paper formula holds with Lm := -A.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  All tensor pointers are DEVICE pointers (HIP global memory of
 *   the current device) owned by the caller; the library allocates no device
 *   memory and keeps no state between calls apart from loaded code objects.
 *   Tensors are dense, row-major and contiguous; every pointer must be
 *   16-byte aligned.  Outputs must not overlap inputs.
 * Layouts.  K [B, L, H, dk], V [B, L, H, dv], W [B, L, H, dk],
 *   U [B, L, H, dv], beta [B, L, H] fp32, g [B, L, H] fp32 (g is the
 *   within-chunk inclusive cumulative sum of the per-token log-decay).
 *   Tile tensors A / Tinv: [B, H, L/C, C, C], so tile t = (b H + h) L/C + chunk,
 *   row i = the later token.  INT8 tiles have the same layout in int8 with one
 *   int32 exponent per tile.
 * dtypes.  GDN_F32 stores fp32 and computes with fp32 MFMA.  GDN_BF16 stores
 *   bf16 and rounds every MFMA operand to bf16 (round to nearest even);
 *   products accumulate in fp32, and sums, identity additions and the
 *   residual are formed in fp32.  beta and g are always fp32.
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Every
 *   call only enqueues work on that stream and returns; results are valid
 *   once the stream has synchronised.  No call synchronises the device.
 *   Calls are thread-safe.
 * Errors.  Return GDN_OK (0) or a negative GDN_ERR_* code.  Arguments are
 *   validated before anything is enqueued, so an error return means nothing
 *   was launched.  GDN_ERR_HIP reports a failed launch (hipGetLastError);
 *   faults inside a kernel surface at the caller's next synchronisation.
 *   n_tiles == 0 (or B == 0) is a no-op returning GDN_OK.
 * Sizes.  C in {16, 32, 64, 128}; L % C == 0; dk, dv in {64, 128};
 *   0 <= N <= C - 1 and 0 <= S <= C - 1 (C = 128: N, S <= 63, see below).
 *   Every launch is one workgroup per tile (per (head, 16-column slice) in
 *   the layer forward's state pass) on a 1-D grid, which HIP bounds by
 *   2^31 - 1 workgroups and 2^32 - 1 work items: a call whose tile count
 *   times its workgroup size (64; 128 for the two-wave C = 128 kernels of
 *   the fused path and the integer inverse; 256 for the C = 128 quantiser
 *   and the state pass) passes 2^32 - 1 returns GDN_ERR_SHAPE before any
 *   launch (at most 67,108,863 tiles of 64 work items).
 *   A batch with L % C != 0 goes through the packed-sequence entry points
 *   (gdn_chunk_wy_fused_varlen, gdn_chunk_forward_varlen) as B sequences of
 *   L tokens each, the last chunk of each a partial one.
 * Non-finite values.  Floating-point entry points: a NaN or infinity in the
 *   strictly lower part of a tile of A (or in a chunk's K, V, beta or g)
 *   reaches that tile's (chunk's) outputs only, never another tile's, and an
 *   inverse is non-finite at least at the entry's own position (T_ij
 *   carries -A_ij).  Which other entries of the tile turn non-finite is not
 *   specified: the kernels set the residual E to its exact value 0 on the
 *   band i - j <= N, where a literal evaluation would carry the NaN.
 *   Entries of A on and above the diagonal are never read.  Integer entry
 *   points require finite inputs.
 */
#ifndef GDNINV_H
#define GDNINV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* 2: the integer quantiser and inverses accept C = 128 (three exponents per
 * tile) and the layer forward's `exact` argument takes the integer inverse
 * modes 2 and 3; every call valid under 1 behaves as before.
 * 3: the integer inverses follow Algorithm 1's operator order with one
 * rounding per operator and the no-clip scale rule (different codes from
 * 2), and gdn_chunk_inverse_neumann_i8 / _i16 take a flags argument. */
#define GDN_ABI_VERSION 3

/* flags of gdn_chunk_inverse_neumann_i8 / _i16: every tensor of the integer
 * inverse holds its unit diagonal inside its codes (the plain form) instead
 * of keeping it exact outside them (the split form, 0). */
#define GDN_INT_PLAIN 1

enum gdn_dtype { GDN_F32 = 0, GDN_BF16 = 1, GDN_I8 = 2 };

enum gdn_status {
  GDN_OK = 0,
  GDN_ERR_NULL = -1,        /* a required pointer is NULL                     */
  GDN_ERR_SHAPE = -2,       /* a size is out of range or L % C != 0           */
  GDN_ERR_PARAM = -3,       /* N or S out of range                            */
  GDN_ERR_DTYPE = -4,       /* unknown or unsupported dtype combination       */
  GDN_ERR_ALIGN = -5,       /* a pointer is not 16-byte aligned               */
  GDN_ERR_ALIAS = -6,       /* an output overlaps an input                    */
  GDN_ERR_HIP = -7,         /* the HIP runtime rejected a launch              */
  GDN_ERR_UNSUPPORTED = -8, /* valid request the library does not implement   */
  GDN_ERR_WORKSPACE = -9    /* the caller's workspace is smaller than needed  */
};

/* Version of this ABI (GDN_ABI_VERSION). */
int gdn_abi_version(void);

/* Static, NUL-terminated description of a status code; never NULL. */
const char* gdn_status_string(int status);

/* Default (N, S) per chunk size: 16 -> (3, 2), 32 -> (3, 4) (Section 4.3),
 * 64 -> (3, 8) (Section 4.1), 128 -> (3, 8) per 64-block (Appendix H), for
 * every arithmetic (the paper measures its integer and floating-point
 * settings at the same orders).  Writes *N, *S; GDN_ERR_SHAPE for other C,
 * GDN_ERR_NULL for NULL outputs. */
int gdn_default_order(int C, int* N, int* S);

/* Build the chunk matrices A (Section 2.1 with the Gated DeltaNet gate):
 *   A[t, i, j] = beta_i (k_i . k_j) exp(g_i - g_j) for i > j, 0 otherwise,
 * with i, j tokens of chunk t.  The gate is evaluated as the exponential of
 * the difference.  K: [B, L, H, dk] in k_dtype (GDN_F32 or GDN_BF16);
 * beta, g: [B, L, H] fp32; A: [B, H, L/C, C, C] in a_dtype (GDN_F32 or
 * GDN_BF16; the upper triangle and diagonal are written as 0).  The Gram
 * product accumulates in fp32. */
int gdn_build_A(const void* K, const float* beta, const float* g, void* A,
                int B, int L, int H, int dk, int C, int k_dtype, int a_dtype,
                void* stream);

/* MatMul-only approximate inverse (Sections 3.1-3.4, Algorithm 1):
 *   T0   = M^(N) (Hadamard) sum_{n=0}^{N} Lm^n,  M^(N)_ij = [i - j <= N],
 *   E    = I - (I + A) T0,
 *   Tinv = T0 sum_{s=0}^{S} E^s            (the ordering of Section 3.4 and
 *                                            Appendix D).
 * A: n_tiles tiles of C x C (entries on/above the diagonal are ignored);
 * Tinv: same shape, written with exact unit diagonal and zero upper
 * triangle.  dtype GDN_F32 or GDN_BF16 for both A and Tinv.  C = 128 is
 * computed block-wise (Appendix E, Appendix H): both 64 x 64 diagonal blocks
 * by the formula above with the given (N, S), joined by
 * Tinv_21 = -Tinv_22 A_21 Tinv_11. */
int gdn_chunk_inverse_neumann(const void* A, void* Tinv, int64_t n_tiles, int C,
                              int N, int S, int dtype, void* stream);

/* Exact inverse (I + A)^-1 by forward substitution (Section 2.2): row by
 * row, n_i = -a_i - a_i N_{0:i,0:i} over the finished rows, Tinv = I + N.
 * Computed in fp32 whatever the storage dtype.  A, Tinv as above. */
int gdn_chunk_inverse_fwdsub(const void* A, void* Tinv, int64_t n_tiles, int C,
                             int dtype, void* stream);

/* Exact inverse (I + A)^-1 with matrix products only: the two-block
 * recursion of Appendix E, X_21 = X_22 L_21 X_11 with L = -A, taken all the
 * way down.  Inside each 16 x 16 diagonal block it runs on masked 16 x 16
 * products (X_{k+1} = X_k + X_k O_k X_k, O_k the entries of L joining blocks
 * of size 2^k); across the 16 x 16 blocks it continues as block forward
 * substitution X_IJ = X_II sum_{K=J}^{I-1} L_IK X_KJ.  C = 128 joins two
 * 64-blocks by Tinv_21 = -Tinv_22 A_21 Tinv_11.  Products in the compute
 * dtype as for gdn_chunk_inverse_neumann (bf16 operands round to bf16).
 * A, Tinv, n_tiles, C, dtype as for gdn_chunk_inverse_neumann. */
int gdn_chunk_inverse_blockwise(const void* A, void* Tinv, int64_t n_tiles, int C, int dtype,
                                void* stream);

/* WY application: per chunk, W = Tinv diag(beta) K and U = Tinv diag(beta) V.
 * Tinv: [B, H, L/C, C, C], K/W: [B, L, H, dk], V/U: [B, L, H, dv], all in
 * `dtype` (GDN_F32 or GDN_BF16); beta fp32.  Only the lower triangle of
 * Tinv is read. */
int gdn_wy_apply(const void* Tinv, const void* K, const void* V, const float* beta,
                 void* W, void* U, int B, int L, int H, int dk, int dv, int C,
                 int dtype, void* stream);

/* Fused path in one launch: gdn_build_A, gdn_chunk_inverse_neumann and
 * gdn_wy_apply with every intermediate kept on chip.  Tinv may be NULL;
 * otherwise the approximate inverse is also written ([B, H, L/C, C, C]).
 * dtype applies to K, V, W, U and Tinv.  A is formed in fp32 and rounded to
 * the compute dtype as an MFMA operand.  C = 128 uses the block form of
 * Appendix E with the 64-row halves 1, 2: W_1 = X_11 diag(beta_1) K_1 and
 * W_2 = X_22 (diag(beta_2) K_2 - A_21 W_1) (the same for U), which equals
 * Tinv diag(beta) K for the block inverse gdn_chunk_inverse_neumann
 * computes; X_21 = -X_22 A_21 X_11 is formed only when Tinv is requested. */
int gdn_chunk_wy_fused(const void* K, const void* V, const float* beta, const float* g,
                       void* W, void* U, void* Tinv, int B, int L, int H, int dk,
                       int dv, int C, int N, int S, int dtype, void* stream);

/* The fused path of gdn_chunk_wy_fused with the exact inverse of
 * gdn_chunk_inverse_blockwise in place of T_hat(N, S): W = X diag(beta) K,
 * U = X diag(beta) V with X = (I + A)^-1 (C = 128 in the same block form as
 * gdn_chunk_wy_fused).  Arguments as gdn_chunk_wy_fused without N, S. */
int gdn_chunk_wy_fused_blockwise(const void* K, const void* V, const float* beta, const float* g,
                                 void* W, void* U, void* Tinv, int B, int L, int H, int dk, int dv,
                                 int C, int dtype, void* stream);

/* gdn_chunk_wy_fused (exact = 0) or gdn_chunk_wy_fused_blockwise (exact = 1)
 * over packed sequences of different lengths: K [1, T, H, dk], V [1, T, H,
 * dv], beta, g [1, T, H] hold the sequences one after another; sequence s
 * is tokens cu_seqlens[s] .. cu_seqlens[s + 1] - 1.  Chunks start at every
 * sequence start, so the last chunk of a sequence holds m = l - C (ceil(l / C)
 * - 1) <= C tokens; it is solved on its m x m system (Section 2.1 with the
 * chunk's tokens only), and g must be the within-chunk cumulative sum for
 * this chunking.  chunk_offsets[s] = sum over r < s of ceil(l_r / C), with
 * chunk_offsets[nseq] = n_chunks.  Both tables are int32 DEVICE arrays of
 * nseq + 1 entries, non-decreasing, cu_seqlens[0] = 0 and
 * cu_seqlens[nseq] <= T; entries inconsistent with them make the affected
 * chunks write nothing (never an access outside the arrays).  W, U:
 * [1, T, H, d], rows of every token written.  Tinv (nullable):
 * [H, n_chunks, C, C], the m x m inverse in the top left of each tile and the
 * identity past m.  C in {16, 32, 64, 128}; C = 128 in the block form of
 * gdn_chunk_wy_fused, a partial chunk as the 128 x 128 tile padded with
 * tokens that write nothing. */
int gdn_chunk_wy_fused_varlen(const void* K, const void* V, const float* beta, const float* g,
                              void* W, void* U, void* Tinv, const int32_t* cu_seqlens,
                              const int32_t* chunk_offsets, int nseq, int n_chunks, int T, int H,
                              int dk, int dv, int C, int N, int S, int exact, int dtype,
                              void* stream);

/* INT8 mode, step 1 (Appendix G quantiser with a power-of-two scale): per
 * tile, Aq = round-half-even(A / 2^e) with e the smallest integer at which
 * every code lies in [-127, 127] (the finest scale at which the clip of
 * q(x) = clip(round(x / Delta)) never acts: max|A| < 127.5 2^e).
 * A: fp32 tiles; Aq: int8 tiles (same layout); eA: int32 [n_tiles].  An
 * all-zero tile gets Aq = 0, eA = 0.  Only the strictly lower part of A is
 * read (the rest is taken as 0 and written as 0).  C in {16, 32, 64, 128}.
 * C = 128 is quantised block-wise (Appendix E with the 64 x 64 blocks of
 * Appendix H): the strict lower parts of the diagonal blocks and the whole
 * block 21 each get their own exponent, eA [n_tiles, 3] in the block order
 * (11, 21, 22); block 12 is written as 0. */
int gdn_quantize_tiles_i8(const float* A, int8_t* Aq, int32_t* eA, int64_t n_tiles,
                          int C, void* stream);

/* INT8 mode, step 2: the approximate inverse of gdn_chunk_inverse_neumann in
 * integer arithmetic (Algorithm 1 with the integer activations of Section
 * 3.5 and Appendix G).  Every tensor is codes with one power-of-two scale
 * per tile; every operator of Algorithm 1 is evaluated exactly from its
 * operands' codes (int8 x int8 MFMA products exact in int32) and its result
 * quantised once by the scale rule of gdn_quantize_tiles_i8:
 *   P_n = q(P_{n-1} Lm), T0 = q(T0 + P_n) (n <= N, P_1 = Lm = -A),
 *   T0 masked once (codes zeroed, scale kept), E = I - q((I + A) T0),
 *   P_s = q(P_{s-1} E), T = q(T + P_s) (s <= S, P_1 = E), Tinv = q(T0 T).
 * flags 0 (split form): the unit diagonal of T0, T and Tinv stays exact
 * outside the codes: Tinv = I + Tq * 2^eT, Tq the strict lower part (0 on
 * and above the diagonal).  GDN_INT_PLAIN (C <= 64): the diagonal is part
 * of every tensor: Tinv = Tq * 2^eT, Tq lower triangular with its diagonal.
 * eT int32 [n_tiles]; Tdeq (nullable) receives Tinv in fp32.  Sums are
 * exact (int32 or fp64) whenever a three-term sum spans at most 52 bits,
 * every tile of the quantiser's output in practice; beyond, a term that
 * cannot move a code is dropped and any other is rounded to the 52-bit
 * window.  C in {16, 32, 64, 128}.  C = 128 runs block-wise (Appendix E,
 * Appendix H) on the codes of gdn_quantize_tiles_i8 at C = 128
 * (eA [n_tiles, 3]): both 64 x 64 diagonal blocks by the integer inverse
 * above (X = I + N per block), and X21 = -X22 A21 X11 as two MatMuls,
 * P = q(A21 + A21 N11), then X21 = -q(P + N22 P); eT [n_tiles, 3] holds the
 * exponents of N11, X21 and N22, so Tinv = I + (each block's codes) *
 * 2^(its exponent), and N, S <= 63.  No code ever saturates (the scale rule
 * leaves the clip inactive), so no saturation count is returned.  Requires
 * finite inputs.  Other flags: GDN_ERR_PARAM; GDN_INT_PLAIN at C = 128:
 * GDN_ERR_UNSUPPORTED. */
int gdn_chunk_inverse_neumann_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq,
                                 int32_t* eT, float* Tdeq, int64_t n_tiles, int C,
                                 int N, int S, int flags, void* stream);

/* INT8 mode in one launch: A in fp32 from K, beta, g (the values
 * gdn_build_A writes with a_dtype GDN_F32), quantised per tile in registers
 * by the rule of gdn_quantize_tiles_i8, then the integer inverse of
 * gdn_chunk_inverse_neumann_i8 (Section 3.5, Appendix G).  K: [B, L, H, dk]
 * in k_dtype (GDN_F32 or GDN_BF16); beta, g: [B, L, H] fp32.  Outputs as
 * gdn_chunk_inverse_neumann_i8, in the [B, H, L/C, C, C] tile order.
 * C in {16, 32, 64, 128}; C = 128 block-wise with eT [n_tiles, 3] (A in
 * fp32 block by block, each block quantised with its own exponent, then the
 * block-wise integer inverse).  Given the same fp32 A tile the codes equal
 * those of gdn_quantize_tiles_i8 followed by gdn_chunk_inverse_neumann_i8. */
int gdn_chunk_inverse_neumann_i8_fused(const void* K, const float* beta, const float* g,
                                       int8_t* Tq, int32_t* eT, float* Tdeq, int B, int L, int H,
                                       int dk, int C, int N, int S, int k_dtype, void* stream);

/* INT16 mode, step 1: the quantiser of gdn_quantize_tiles_i8 with 16-bit
 * codes (Appendix G lists INT16 activations for the inverse): per tile,
 * Aq = round-half-even(A / 2^e) with e the smallest integer at which every
 * code lies in [-32639, 32639].  A: fp32 tiles; Aq: int16 tiles (same
 * layout); eA: int32 [n_tiles].  An all-zero tile gets Aq = 0, eA = 0.  Only
 * the strictly lower part of A is read (the rest is taken as 0 and written
 * as 0).  C = 128: block-wise with eA [n_tiles, 3], as for
 * gdn_quantize_tiles_i8. */
int gdn_quantize_tiles_i16(const float* A, int16_t* Aq, int32_t* eA, int64_t n_tiles,
                           int C, void* stream);

/* INT16 mode, step 2: the integer inverse of gdn_chunk_inverse_neumann_i8
 * with 16-bit codes (Section 3.5): codes in [-32639, 32639] (32639 =
 * 127 * 256 + 127), every product exact (each code split into two int8
 * limbs, four int8 MFMAs per product, recombined exactly in fp64), every
 * operator's result quantised once to 16 bits by the scale rule of
 * gdn_quantize_tiles_i16; order, forms (flags), outputs and the exactness
 * statement as gdn_chunk_inverse_neumann_i8, with int16 Tq.  Aq codes must
 * lie in [-32639, 32639], the range the quantiser writes (a negated code
 * must split into two int8 limbs); a tile holding -32768 gets unspecified
 * codes.  C in {16, 32, 64, 128}; C = 128 block-wise with eA, eT
 * [n_tiles, 3], as for gdn_chunk_inverse_neumann_i8. */
int gdn_chunk_inverse_neumann_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq,
                                  int32_t* eT, float* Tdeq, int64_t n_tiles, int C,
                                  int N, int S, int flags, void* stream);

/* The forward-substitution baseline in INT16 (the integer counterpart of
 * gdn_chunk_inverse_fwdsub, beside the integer Neumann inverse): Section
 * 2.2's recurrence x_ij = -a_ij - sum_{j<k<i} a_ik x_kj run row by row on
 * 16-bit codes with one power-of-two exponent per tile (the per-tensor
 * scheme of Appendix G).  Row i is the sum of -a_i (codes at eA) and
 * -a_i X (exact products at eA + eT), aligned 16 guard bits under a code's
 * quantum (finer product terms rounded half-even to that grid); the tile
 * exponent eT starts at eA and
 * grows by the smallest shift that fits a new row (earlier rows rounded
 * half-even to it); the row's codes are one half-even rounding of its sum.
 * Aq, eA as for gdn_chunk_inverse_neumann_i16 (codes in [-32639, 32639]);
 * outputs Tq, eT, Tdeq (nullable) likewise.  C in {16, 32, 64}. */
int gdn_chunk_inverse_fwdsub_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq,
                                 int32_t* eT, float* Tdeq, int64_t n_tiles, int C,
                                 void* stream);

/* The same forward substitution on 8-bit codes (the integer baseline beside
 * gdn_chunk_inverse_neumann_i8): codes in [-127, 127], sum terms aligned
 * below 2^23, with the arguments and layouts of gdn_chunk_inverse_neumann_i8
 * (without N, S). */
int gdn_chunk_inverse_fwdsub_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                                float* Tdeq, int64_t n_tiles, int C, void* stream);

/* INT16 mode in one launch: A in fp32 from K, beta, g (the values
 * gdn_build_A writes with a_dtype GDN_F32), quantised per tile in registers
 * by the rule of gdn_quantize_tiles_i16, then the integer inverse of
 * gdn_chunk_inverse_neumann_i16.  Arguments and layouts as
 * gdn_chunk_inverse_neumann_i8_fused, with int16 Tq (C = 128 block-wise with
 * eT [n_tiles, 3]).  Given the same fp32 A tile the codes equal those of
 * gdn_quantize_tiles_i16 followed by gdn_chunk_inverse_neumann_i16. */
int gdn_chunk_inverse_neumann_i16_fused(const void* K, const float* beta, const float* g,
                                        int16_t* Tq, int32_t* eT, float* Tdeq, int B, int L,
                                        int H, int dk, int C, int N, int S, int k_dtype,
                                        void* stream);

/* Chunk-wise Gated DeltaNet forward of one layer, built around the chunk
 * inverse: the chunk-level recurrence of Gated DeltaNet that Section 1
 * starts from, with Y = T^-1 X (Appendix E) evaluated per chunk.  Per head,
 * with the [dk, dv] state S, the token recurrence it computes is
 *   S_t = a_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T,
 *   o_t = scale S_t^T q_t,   a_t = exp(g_t - g_{t-1}) inside a chunk,
 * evaluated chunk by chunk: T = (I + A)^-1 chosen by `exact` (the inverse
 * mode): 0, T_hat(N, S) of gdn_chunk_inverse_neumann; 1, the exact
 * block-wise inverse; 2 and 3, the quantised GDN of Section 3.5: T_hat(N, S)
 * in integer arithmetic on 16-bit (2) or 8-bit (3) codes, the codes of
 * gdn_chunk_inverse_neumann_i16_fused (_i8_fused) for the chunk, dequantised
 * to fp32 (modes 2 and 3 run the default (N, S) of gdn_default_order with
 * dk = dv = 128, else GDN_ERR_UNSUPPORTED; any other mode GDN_ERR_PARAM),
 * W = T diag(beta e^g) K, U = T diag(beta) V, V_new = U - W S,
 * O = scale (diag(e^g) Q S + ((Q K^T) (.) D) V_new) with D_ij = e^{g_i - g_j}
 * for i >= j (else 0), S' = e^{g_last} S + K^T diag(e^{g_last - g}) V_new.
 * Q, K: [B, L, H, dk]; V, O: [B, L, H, dv], all in `dtype` (GDN_F32 or
 * GDN_BF16); beta, g: [B, L, H] fp32 as for gdn_build_A.  S0 (nullable:
 * zero state) and S_final (nullable: not written): [B, H, dk, dv] fp32;
 * S_final may be S0 itself (updated in place) but must not overlap it
 * otherwise.  bf16 mode rounds to bf16 every MFMA operand, including the
 * state where it multiplies W and Q and V_new where it multiplies P and K^T;
 * the state itself is carried in fp32.  workspace: device memory of at least
 * gdn_chunk_forward_workspace() bytes, owned by the caller, contents
 * undefined on return; it must not overlap any tensor argument.
 * C in {16, 32, 64} (GDN_ERR_UNSUPPORTED for 128).  L = 0 with B H > 0
 * copies S0 (or zeros) into S_final.  GDN_ERR_WORKSPACE if workspace_bytes
 * is too small.  Two launches on `stream`: every chunk in parallel, then one
 * wave per (batch, head, 16 value columns) walking the chunks in order. */
int gdn_chunk_forward(const void* Q, const void* K, const void* V, const float* beta,
                      const float* g, const float* S0, void* O, float* S_final, void* workspace,
                      int64_t workspace_bytes, int B, int L, int H, int dk, int dv, int C, int N,
                      int S, int exact, float scale, int dtype, void* stream);

/* gdn_chunk_forward in its two phases, for callers that schedule them apart
 * (the first has no sequential dependence; the second carries the state).
 * gdn_chunk_forward_prepare: every chunk in parallel, Q, K, V, beta, g ->
 * workspace (T by the inverse mode `exact` as for gdn_chunk_forward, then
 * the per-chunk factors).  gdn_chunk_forward_state: the recurrence over the
 * chunks of each head, workspace (as the prepare call with the same sizes
 * and dtype left it), Q, g, S0 -> O, S_final.  Run on one stream, prepare
 * then state equals gdn_chunk_forward bit for bit.  Arguments, layouts and
 * errors as for gdn_chunk_forward; the prepare call does not read S0 and
 * writes neither O nor S_final. */
int gdn_chunk_forward_prepare(const void* Q, const void* K, const void* V, const float* beta,
                              const float* g, void* workspace, int64_t workspace_bytes, int B,
                              int L, int H, int dk, int dv, int C, int N, int S, int exact,
                              int dtype, void* stream);
int gdn_chunk_forward_state(const void* Q, const float* g, const float* S0, void* O,
                            float* S_final, const void* workspace, int64_t workspace_bytes, int B,
                            int L, int H, int dk, int dv, int C, float scale, int dtype,
                            void* stream);

/* gdn_chunk_forward without a caller's workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): the workspace between the two
 * launches is a file-scope device array of GDN_FORWARD_SCRATCH_BYTES that
 * every device the library runs on holds until the process ends (looked up
 * on the first call on a device); the call itself allocates nothing.
 * Arguments, layouts, results (bit for bit) and errors as for
 * gdn_chunk_forward without workspace and workspace_bytes; sizes whose
 * workspace (gdn_chunk_forward_workspace) exceeds the array return
 * GDN_ERR_WORKSPACE before any HIP call (bf16: 2048 chunk tiles of
 * C = 64, dk = dv = 128 fit).  Every call on a device shares that device's
 * array: calls that overlap in time on one device (two streams, two host
 * threads) race and must be serialised by the caller.  The array keeps the
 * last call's contents; nothing in it needs to start at zero (each call's
 * first launch writes every byte its second launch reads). */
#define GDN_FORWARD_SCRATCH_BYTES ((int64_t)128 << 20)
int gdn_chunk_forward_noalloc(const void* Q, const void* K, const void* V, const float* beta,
                              const float* g, const float* S0, void* O, float* S_final, int B,
                              int L, int H, int dk, int dv, int C, int N, int S, int exact,
                              float scale, int dtype, void* stream);

/* Workspace bytes gdn_chunk_forward needs for these sizes (0 when there is
 * no chunk); GDN_ERR_SHAPE / GDN_ERR_DTYPE / GDN_ERR_NULL as for the call. */
int gdn_chunk_forward_workspace(int B, int L, int H, int dk, int dv, int C, int dtype,
                                int64_t* bytes);

/* The layer forward of gdn_chunk_forward over packed variable-length
 * sequences (the layouts and chunk tables of gdn_chunk_wy_fused_varlen):
 * every sequence runs the chunk-wise recurrence from its own initial state,
 * its chunks starting at its first token; a last chunk of m < C tokens is
 * the m x m system (its rows past m are neither read for output nor
 * written).  Q, K: [1, T, H, dk]; V, O: [1, T, H, dv] in `dtype`; beta, g:
 * [1, T, H] fp32 (g the within-chunk cumulative log-decay for this
 * chunking).  S0, S_final (nullable; S_final may equal S0):
 * [nseq, H, dk, dv] fp32, the state of every (sequence, head); an empty
 * sequence keeps its initial state.  workspace: at least the bytes
 * gdn_chunk_forward_workspace reports for B = 1, L = n_chunks * C.  The
 * per-chunk launch and the state pass run back to back on `stream`.
 * Inverse modes (`exact`) as for gdn_chunk_forward; in the integer modes a
 * partial chunk is the C x C tile padded with tokens that write nothing.
 * C in {16, 32, 64}. */
int gdn_chunk_forward_varlen(const void* Q, const void* K, const void* V, const float* beta,
                             const float* g, const float* S0, void* O, float* S_final,
                             void* workspace, int64_t workspace_bytes,
                             const int32_t* cu_seqlens, const int32_t* chunk_offsets, int nseq,
                             int n_chunks, int T, int H, int dk, int dv, int C, int N, int S,
                             int exact, float scale, int dtype, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GDNINV_H */
