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

// Decode GEMM geometry: a workgroup owns 16 output columns over the whole K
// range (no cross-workgroup reduction); its waves split K; one MFMA tile has
// 16 rows of M; one launch handles up to 4 row tiles.
constexpr int kTileN = 16;
constexpr int kTileM = 16;
constexpr int kDecodeMaxM = 64;
// Largest LDS a decode workgroup may use (gfx950 has 160 KB per CU).
constexpr size_t kLdsMax = 160 * 1024;

// How a decode kernel obtains each row's scale and zero.
enum MetaMode {
  kMetaGroup = 0,      // sorted rows: one (scale, zero) per 32-row step, staged in LDS
  kMetaRowGlobal = 1,  // per row through g_idx, read from global memory (Fig. 1 as drawn)
  kMetaRowLds = 2,     // per row through g_idx, tile metadata staged in LDS
};
// Where the A operand (activations) comes from.
enum AMode {
  kAGlobal = 0,        // 16-byte fragment loads from global memory, permuted in registers
  kALds = 1,           // whole X staged in LDS in operand order
  kALdsGather = 2,     // X[:, perm] gathered into LDS in operand order
  kAGlobalPrep = 3,    // 16-byte fragment loads of an operand already in operand order
};
// What the caller hands the GEMM as its activations.
enum Operand {
  kOperandPlain = 0,     // X row-major
  kOperandGather = 1,    // X row-major, used as X[:, perm]
  kOperandPrepared = 2,  // X[:, perm] already gathered and in operand order (k_gather_prep)
};

// One decode launch (device pointers).
struct GemmArgs {
  const uint16_t* X;      // [M][ldx] fp16 bits
  int64_t ldx;
  int M;
  const int32_t* perm;    // kALdsGather: column j of the operand is column perm[j] of X
  const uint32_t* qw;     // GPTQ: [K/8][ldq]; tiled: [ceil(N/16)][ldq]
  int64_t ldq;
  const uint16_t* sc;     // [num_groups][lds]
  int64_t lds;
  const uint32_t* qz;     // [num_groups][ldz]
  int64_t ldz;
  const int32_t* g_idx;   // [K] (per-row metadata modes)
  int K, N, G, num_groups;
  int zoff;      // added to every stored zero code (the layer's zero_offset)
  int ks;        // M-tiled kernel: K splits (<= 1: none)
  float* part;   // M-tiled kernel: fp32 partials [ks][M][N] when ks > 1
  int dt;        // tpdq_dtype of X, scales and Y (the kernels take it as a template argument)
  uint16_t* Y;            // [M][ldy]
  int64_t ldy;
  // optional second copy of Y in the prepared-operand layout of a GEMM whose K
  // is this N (k_ordered and k_rowmeta; N % 128 == 0), natural order when
  // that GEMM's weights are tiled
  uint16_t* Yp;
  int yp_natural;
  // gated GEMM (plan.gated): the up projection's weights and metadata, with
  // the same shape, leading dimensions, g_idx and layout as qw, sc, qz
  const uint32_t* qw_up;
  const uint16_t* sc_up;
  const uint32_t* qz_up;
  int meta_rows;          // metadata rows staged in LDS
  int lds_x_off;          // byte offset of the staged X in LDS
  int lds_xr_off;         // kALdsGather: byte offset of the LDS copy of X's rows
};

// Host-side plan of one decode launch.
struct DecodePlan {
  bool gated;   // Y = silu(X W) * (X W_up): two weight streams, tn = 2
  int dt;       // tpdq_dtype
  int layout;   // tpdq_layout of qweight
  int meta;     // MetaMode
  int amode;    // AMode
  int nw;       // waves per workgroup
  int mt;       // row tiles (1, 2, 4)
  int tn;       // 16-column tiles per workgroup (ordered kernel: 1 or 2)
  int spg;      // 32-row steps per group (kMetaGroup)
  int meta_rows;
  size_t lds_bytes;
  int lds_x_off;
  int lds_xr_off;
  bool wide;    // k_wide: waves over columns, X shared through LDS in chunks
  int ks;       // k_wide: K splits (fp32 partials, then k_splitk_reduce)
};
// k_wide: 8 waves (128 columns) per workgroup; used on weights of at least
// kWideMinWeights elements when X does not fit in LDS, K split until about
// kWideTargetWgs workgroups stream.
constexpr int kWideWaves = 8;
constexpr int64_t kWideMinWeights = (int64_t)64 << 20;
// ... and from 16M elements when X is row-major with four row tiles
// (M > 32), or two with K >= N: the tile kernel's loads of row-major X then
// touch 16 rows a row apart per instruction, which the wide kernel's staging
// avoids (with two row tiles and K < N the tile kernel stays faster)
constexpr int64_t kWideMinWeightsRowMajor = (int64_t)16 << 20;
constexpr int kWideTargetWgs = 200;

// The in-LDS gather of X[:, perm] is planned on grids of at most this many
// 16-column tiles; on larger ones (the unsharded Llama-70B GEMM1: 1792 tiles,
// each workgroup loading the 32 KiB permutation and X) the caller gathers X'
// once, row-major, and the kernel stages it like any X (MLP at M = 1:
// 50.1 -> 48.4 us; at TP = 8, 224 tiles, the in-LDS gather stays: 0.9 us)
constexpr int kGatherOnceTiles = 512;
// meta_pref: kMetaGroup for sorted rows (needs G % 32 == 0), otherwise a
// per-row mode; operand: an Operand. Returns false when no decode kernel
// covers the request (for kOperandGather: the gather is not planned inside
// the kernel, the caller then gathers X' first, row-major (launch_gather_plain,
// planning with kOperandPlain) or in operand order (launch_gather_prep,
// kOperandPrepared)).
bool plan_decode(int M, int K, int N, int G, int num_groups, int layout, int meta_pref, int operand,
                 int dt, DecodePlan* p, bool gated = false);
// the kernel of a plan, per element type (gemm_decode.hip, gemm_decode_bf16.hip)
typedef void (*DecodeKernel)(GemmArgs);
DecodeKernel decode_kernel_f16(const DecodePlan& p);
DecodeKernel decode_kernel_bf16(const DecodePlan& p);
DecodeKernel decode_kernel_gated_f16(const DecodePlan& p);   // gemm_gated.hip
DecodeKernel decode_kernel_gated_bf16(const DecodePlan& p);  // gemm_gated_bf16.hip
// part: the workspace for k_wide's split-K partials (ks x M x N floats)
hipError_t launch_decode(const GemmArgs& a, const DecodePlan& p, float* part, hipStream_t s);
// Xp [M][K] = X[:, perm] row-major (perm required).
hipError_t launch_gather_plain(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                               uint16_t* Xp, hipStream_t s);
// Xp [M][K] = X[:, perm] (perm may be NULL), each octet in operand order.
hipError_t launch_gather_prep(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                              int layout, uint16_t* Xp, hipStream_t s);

// M-tiled MFMA GEMM (gemm_prefill.hip): sorted rows, tiled weights. At
// M >= kPrefillMinM, 128 x 512 tiles over the whole K; from kMtileMinM rows,
// on weights of at least kMtileMinWeights elements, 64 x 512 tiles with K
// split over ks workgroups (fp32 partials in the workspace, summed in split
// order by a second kernel). Below kMtileMinM rows the decode kernels are
// faster (measured on the Llama-70B TP=1 shapes: at M = 16 the decode GEMMs
// take 38 / 34 us, the split-K tiles 57 / 61 us; at M = 64, 127 / 111 us
// against 70 / 64 us).
constexpr int kPrefillMinM = 256;
constexpr int kMtileMinM = 33;
constexpr int64_t kMtileMinWeights = (int64_t)64 << 20;
constexpr int kMtileSlots = 256;  // one 8-wave workgroup per CU on 256 CUs
struct MtilePlan {
  int rt, nw, st, ks;  // row tiles and waves per workgroup, LDS stages, K splits
};
bool plan_mtile(int M, int64_t ldx, const tpdq_w4* w, int meta, MtilePlan* p);
// workspace bytes of the fp32 partials (0 when ks == 1)
size_t mtile_part_bytes(const MtilePlan& p, int M, int N);
// part: the partials (ignored when p.ks == 1)
hipError_t launch_mtile(const GemmArgs& a, const MtilePlan& p, float* part, hipStream_t s);
hipError_t launch_splitk_reduce(const float* part, int ks, int M, int N, uint16_t* Y, int64_t ldy,
                                int dt, hipStream_t s);
// Xp [M][K] = X[:, perm] row-major (for the prefill GEMM's activations)
hipError_t launch_gather_rows(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
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
// offs: the group counts of launch_gidx_validate, turned into each group's
// first sorted row (an exclusive scan, in place) before the ranking
hipError_t launch_gidx_rank(const ReorderLayer& L, uint32_t* offs, hipStream_t s);
// dst = src[Prow, Pcol] (either permutation may be NULL = identity), src in
// GPTQ layout, dst dense in dst_layout.
hipError_t launch_permute_qweight(const uint32_t* src, int64_t ld_src, int K, int N,
                                  const int32_t* Prow, const int32_t* Pcol, uint32_t* dst,
                                  int dst_layout, hipStream_t s);
// words per 16-column tile of a dense tiled qweight with K rows
__host__ __device__ inline int64_t tiled_ld(int K) { return (int64_t)((K + 127) / 128) * 256; }
hipError_t launch_permute_scales(const uint16_t* src, int64_t ld_src, int ng, int N,
                                 const int32_t* Pcol, uint16_t* dst, hipStream_t s);
hipError_t launch_permute_qzeros(const uint32_t* src, int64_t ld_src, int ng, int N,
                                 const int32_t* Pcol, uint32_t* dst, hipStream_t s);

}  // namespace tpdq
