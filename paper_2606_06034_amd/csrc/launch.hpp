// launch.hpp -- host-side launchers behind the C ABI (internal).
// Every launcher assumes validated arguments, enqueues on `st` and returns
// hipGetLastError() (hipErrorNotSupported for combinations not built).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

// compile-time feature widths for the templated launchers
#define GDN_DK_SWITCH(dk, ...)                     \
  switch (dk) {                                    \
    case 64: { constexpr int DK = 64; __VA_ARGS__ }   \
    case 128: { constexpr int DK = 128; __VA_ARGS__ } \
  }
#define GDN_DV_SWITCH(dv, ...)                     \
  switch (dv) {                                    \
    case 64: { constexpr int DV = 64; __VA_ARGS__ }   \
    case 128: { constexpr int DV = 128; __VA_ARGS__ } \
  }

// Waves per workgroup of the fused kernel (Chunk::grouped; packed sequences:
// consecutive work items): 4 when 32 divides H, 2 when 16 does, else 1.  A
// workgroup then covers a 1 KB (512 B) run of every token row of its chunk,
// which the long-context shape runs at 0.69 of HBM instead of 0.59 with one
// wave per workgroup.
inline int waves_per_group(int H) {
  return (H % 32 == 0) ? 4 : (H % 16 == 0) ? 2 : 1;
}

hipError_t launch_neumann(const void* A, void* T, int64_t n_tiles, int C, int N, int S,
                          int dtype, hipStream_t st);
hipError_t launch_fwdsub(const void* A, void* T, int64_t n_tiles, int C, int dtype,
                         hipStream_t st);
hipError_t launch_blockwise(const void* A, void* T, int64_t n_tiles, int C, int dtype,
                            hipStream_t st);
hipError_t launch_build_A(const void* K, const float* beta, const float* g, void* A, int B,
                          int L, int H, int dk, int C, int k_dtype, int a_dtype, hipStream_t st);
hipError_t launch_wy(const void* T, const void* K, const void* V, const float* beta, void* W,
                     void* U, int B, int L, int H, int dk, int dv, int C, int dtype,
                     hipStream_t st);
// exact: the exact block-wise inverse instead of T_hat(N, S)
hipError_t launch_fused(const void* K, const void* V, const float* beta, const float* g, void* W,
                        void* U, void* T, int B, int L, int H, int dk, int dv, int C, int N,
                        int S, int dtype, bool exact, hipStream_t st);
// chunk-wise Gated DeltaNet forward; ws holds fwd_workspace_elems(C, dk, dv)
// elements of the IO type per chunk tile.  phases: bit 0 the per-chunk
// launch (Q, K, V, beta, g -> ws), bit 1 the state pass (ws, Q, g, S0 -> O,
// S_final)
hipError_t launch_forward(const void* Q, const void* K, const void* V, const float* beta,
                          const float* g, const float* S0, void* O, float* Sfin, void* ws, int B,
                          int L, int H, int dk, int dv, int C, int N, int S, int mode,
                          float scale, int dtype, int phases, hipStream_t st);
hipError_t launch_forward_varlen(const void* Q, const void* K, const void* V, const float* beta,
                                 const float* g, const float* S0, void* O, float* Sfin, void* ws,
                                 const int* cu, const int* off, int nseq, int nchunks, int Ttok,
                                 int H, int dk, int dv, int C, int N, int S, int mode,
                                 float scale, int dtype, hipStream_t st);
int64_t fwd_workspace_elems(int C, int dk, int dv);
// the fused kernel over packed sequences (C <= 64): cu, off device tables of
// nseq + 1 token / chunk offsets, nchunks chunks, Ttok tokens
hipError_t launch_fused_varlen(const void* K, const void* V, const float* beta, const float* g,
                               void* W, void* U, void* T, const int* cu, const int* off, int nseq,
                               int nchunks, int Ttok, int H, int dk, int dv, int C, int N, int S,
                               int dtype, bool exact, hipStream_t st);
hipError_t launch_quantize_i8(const float* A, int8_t* Aq, int32_t* eA, int64_t n_tiles, int C,
                              hipStream_t st);
hipError_t launch_neumann_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                             float* Tdeq, int64_t n_tiles, int C, int N, int S, bool plain,
                             hipStream_t st);
hipError_t launch_inverse_i8_fused(const void* K, const float* beta, const float* g, int8_t* Tq,
                                   int32_t* eT, float* Tdeq, int B, int L, int H, int dk, int C,
                                   int N, int S, int k_dtype, hipStream_t st);
hipError_t launch_quantize_i16(const float* A, int16_t* Aq, int32_t* eA, int64_t n_tiles, int C,
                               hipStream_t st);
hipError_t launch_neumann_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq, int32_t* eT,
                              float* Tdeq, int64_t n_tiles, int C, int N, int S, bool plain,
                              hipStream_t st);
hipError_t launch_fwdsub_i16(const int16_t* Aq, const int32_t* eA, int16_t* Tq, int32_t* eT,
                             float* Tdeq, int64_t n_tiles, int C, hipStream_t st);
hipError_t launch_fwdsub_i8(const int8_t* Aq, const int32_t* eA, int8_t* Tq, int32_t* eT,
                            float* Tdeq, int64_t n_tiles, int C, hipStream_t st);
hipError_t launch_inverse_i16_fused(const void* K, const float* beta, const float* g,
                                    int16_t* Tq, int32_t* eT, float* Tdeq, int B, int L, int H,
                                    int dk, int C, int N, int S, int k_dtype, hipStream_t st);

// the allocation-free layer forward's scratch: its size, and its device
// address on the current device (looked up once per device)
constexpr int64_t kForwardScratchBytes = int64_t(128) << 20;
hipError_t forward_scratch(void** ptr);

}  // namespace gdn
