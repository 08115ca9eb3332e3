// Internal declarations shared by the host-side translation units of libtpdq.
// Device code lives in the .hip files; this header only carries plain launch
// descriptions, so the ABI layer can validate and dispatch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/tpdq.h"

namespace tpdq {

// Byte offsets inside a caller-supplied workspace are rounded to this.
constexpr size_t kWsAlign = 256;
inline size_t align_up(size_t x, size_t a = kWsAlign) { return (x + a - 1) / a * a; }

// Columns covered by one decode workgroup (4 waves share one column tile and
// split its K range); each lane owns 4 consecutive columns.
constexpr int kDecodeCols = 64;
constexpr int kDecodeWaves = 4;
// Rows of the MFMA tile (v_mfma_f32_16x16x32_f16) and the largest M handled
// by one decode launch (4 row tiles).
constexpr int kTileM = 16;
constexpr int kDecodeMaxM = 64;

// One GEMM launch as the decode kernels see it (device pointers).
struct GemmArgs {
  const uint16_t* X;      // [M][ldx] fp16/bf16 bits
  int64_t ldx;
  int M;
  const uint32_t* qw;     // [K/8][ldq]
  int64_t ldq;
  const uint16_t* sc;     // [num_groups][lds]
  int64_t lds;
  const uint32_t* qz;     // [num_groups][ldz]
  int64_t ldz;
  const int32_t* g_idx;   // [K] (act-order only)
  int K, N, G, num_groups;
  uint16_t* Y;            // [M][ldy]
  int64_t ldy;
  float* partials;        // [splits][M][N] fp32, when splits > 1
  uint32_t* counters;     // [ceil(N/64)], zero on entry and on exit
  int splits;
};

// Split-K factor the decode launch uses for this shape (one place, so the
// workspace query and the launch agree).
int decode_splits(int M, int K, int N);
// Workspace bytes for one decode GEMM (counters + partials), M <= 64.
size_t decode_ws_bytes(int M, int K, int N);

// Launchers (device code in gemm_decode.hip). They return hipSuccess or the
// launch error.
hipError_t launch_decode_ordered(const GemmArgs& a, hipStream_t s);
hipError_t launch_decode_rowmeta(const GemmArgs& a, bool actorder, hipStream_t s);
hipError_t launch_gather_cols(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                              uint16_t* Xp, hipStream_t s);

// Reorder (device code in reorder.hip).
struct ReorderLayer {
  const int32_t* g_idx;
  int K, G, num_groups;
  int32_t* P;
  int32_t* g_sorted;
};
hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t s);
hipError_t launch_gidx_validate(const ReorderLayer& L, uint32_t* counts, uint32_t* flag, hipStream_t s);
hipError_t launch_gidx_rank(const ReorderLayer& L, hipStream_t s);
hipError_t launch_permute_qweight(const uint32_t* src, int64_t ld_src, int K, int N,
                                  const int32_t* Prow, const int32_t* Pcol, uint32_t* dst,
                                  hipStream_t s);
hipError_t launch_permute_scales(const uint16_t* src, int64_t ld_src, int ng, int N,
                                 const int32_t* Pcol, uint16_t* dst, hipStream_t s);
hipError_t launch_permute_qzeros(const uint32_t* src, int64_t ld_src, int ng, int N,
                                 const int32_t* Pcol, uint32_t* dst, hipStream_t s);

}  // namespace tpdq
