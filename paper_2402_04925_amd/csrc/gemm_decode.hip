// Planning and launch of the decode GEMMs (M <= 64), and the gather of the
// activations into decode operand order. The kernels are in decode_kernels.h;
// this file instantiates them for fp16, gemm_decode_bf16.hip for bf16.
#include "decode_kernels.h"

#include <algorithm>

namespace tpdq {
namespace {

// The prepared operand: X'[m][k] = X[m][perm[k]] (perm NULL: X itself) as
// 16-byte records [row tile t][step s][lane l]: row 16 t + l % 16, operand
// rows 8 (4 s + l / 16) .. +7 in operand order (natural for tiled weights,
// x0, x4, x1, x5, ... for GPTQ ones), zero past M or K. A decode wave reads one step of one row tile as one
// contiguous KiB.
// X'[m][k] = X[m][perm[k]] row-major [M][K], one octet per thread: for a
// decode GEMM that then stages X' in LDS (or reads it row-major) like any X.
__global__ __launch_bounds__(64) void k_gather_plain(const uint16_t* __restrict__ X, int64_t ldx,
                                                     int M, int K, const int32_t* __restrict__ perm,
                                                     uint16_t* __restrict__ Xp) {
  const int kw = K >> 3;
  const int64_t total = (int64_t)M * kw;
  const uint32_t kmax = (uint32_t)(K - 1);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(i / kw);
    const int r = (int)(i - (int64_t)m * kw);
    const uint16_t* xr = X + (int64_t)m * ldx;
    const u4_t p0 = *(const u4_t*)(perm + r * 8);
    const u4_t p1 = *(const u4_t*)(perm + r * 8 + 4);
    uint32_t x[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = xr[min(p0[e], kmax)];
      x[e + 4] = xr[min(p1[e], kmax)];
    }
    *(u4_t*)(Xp + (int64_t)m * K + 8 * r) =
        u4_t{x[0] | (x[1] << 16), x[2] | (x[3] << 16), x[4] | (x[5] << 16), x[6] | (x[7] << 16)};
  }
}

__global__ __launch_bounds__(64) void k_gather_prep(const uint16_t* __restrict__ X, int64_t ldx,
                                                    int M, int K, const int32_t* __restrict__ perm,
                                                    int natural, uint16_t* __restrict__ Xp) {
  const int kw = K >> 3;
  const int nsteps = 4 * ((K + 127) >> 7);
  const int mt = (M + kTileM - 1) / kTileM;
  const int64_t total = (int64_t)mt * nsteps * 64;
  const uint32_t kmax = (uint32_t)(K - 1);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int l = (int)(i & 63);
    const int ts = (int)(i >> 6);
    const int t = ts / nsteps;
    const int st = ts - t * nsteps;
    const int m = t * kTileM + (l & 15);
    const int r = 4 * st + (l >> 4);
    u4_t v = {0u, 0u, 0u, 0u};
    if (m < M && r < kw) {
      const uint16_t* xr = X + (int64_t)m * ldx;
      uint32_t c[8];
      if (perm) {
        const u4_t p0 = *(const u4_t*)(perm + r * 8);
        const u4_t p1 = *(const u4_t*)(perm + r * 8 + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          c[e] = min(p0[e], kmax);
          c[e + 4] = min(p1[e], kmax);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) c[e] = (uint32_t)(r * 8 + e);
      }
      uint32_t x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = xr[c[e]];
      v = natural ? u4_t{x[0] | (x[1] << 16), x[2] | (x[3] << 16), x[4] | (x[5] << 16), x[6] | (x[7] << 16)}
                  : u4_t{x[0] | (x[4] << 16), x[1] | (x[5] << 16), x[2] | (x[6] << 16), x[3] | (x[7] << 16)};
    }
    *(u4_t*)(Xp + i * 8) = v;
  }
}

}  // namespace

DecodeKernel decode_kernel_f16(const DecodePlan& p) { return pick_kernel_dt<kF16>(p); }

namespace {
DecodeKernel decode_kernel(const DecodePlan& p) {
  if (p.gated) return p.dt == kBF16 ? decode_kernel_gated_bf16(p) : decode_kernel_gated_f16(p);
  return p.dt == kBF16 ? decode_kernel_bf16(p) : decode_kernel_f16(p);
}
}  // namespace

bool plan_decode(int M, int K, int N, int G, int num_groups, int layout, int meta_pref, int operand,
                 int dt, DecodePlan* p, bool gated) {
  if (M < 1 || M > kDecodeMaxM) return false;
  const int mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  const int ntiles = (N + kTileN - 1) / kTileN;
  // waves per workgroup (the per-row kernels): about 16 resident waves per
  // CU over the grid; the ordered kernel is set below
  int nw = 16;
  if (ntiles > 256) nw = 8;
  if (ntiles > 1024) nw = 4;

  int meta = meta_pref;
  const int spg = G / 32;
  if (meta == kMetaGroup &&
      (G <= 0 || G % 32 != 0 || !(spg == 1 || spg == 2 || spg == 4 || spg == 8)))
    meta = kMetaRowLds;  // sorted rows of another G: per-row groups floor(k / G)
  if ((meta != kMetaGroup || mt == 4) && nw > 8) nw = 8;
  if (meta != kMetaGroup && mt == 4) nw = 4;  // four row tiles of per-row dequant: registers
  if (gated && nw > 8) nw = 8;                 // two weight streams per wave
  // tile metadata in LDS: the per-row act-order kernel only (the ordered
  // kernel's travels with its weight stream)
  int meta_rows = meta == kMetaRowLds ? num_groups : 0;
  const size_t red = (size_t)nw * mt * (gated ? 2 : 1) * 1024;
  size_t meta_bytes =
      meta_rows ? align_up(((size_t)meta_rows * kTileN + 1) * 16, 16) : 0;  // + a spare entry
  if (meta_bytes > kLdsMax - red) {
    meta = kMetaRowGlobal;
    meta_rows = 0;
    meta_bytes = 0;
  }
  // padded X + the zero entry + a spare entry
  const size_t x_bytes = ((size_t)M * 16 * ((K + 127) / 128) + 2) * 16;
  // the gather's copy of X + spare: row-major, or column-major with four
  // halves per column for 2 <= M <= 4 (see XStage)
  const size_t xr_bytes = (M >= 2 && M <= 4) ? (size_t)(K / 8 + 1) * 64
                                             : align_up((size_t)M * K * 2, 16) + 16;
  // stage X in LDS when it leaves room for two workgroups per CU (or one,
  // when the grid has no more workgroups than CUs); the ordered kernel only
  // up to 4 rows: from 8 rows on X read from global memory (two column
  // tiles per workgroup on large grids) measured faster (Llama-70B TP=8 at
  // M = 8: GEMM2 8.43 -> 6.26 us, GEMM1 8.74 -> 8.24 us; at M = 4 LDS wins,
  // GEMM1 6.33 against 7.93 us)
  const size_t budget = ntiles <= 256 ? kLdsMax : kLdsMax / 2;
  // On weights of kWideMinWeights or more, from 3 rows on, the wide kernel
  // (X shared by 8 column tiles through LDS) beats staging all of X per
  // 16-column workgroup (Llama-70B TP=1 GEMM1 at M = 4: 31.0 -> 24.7 us; at
  // M <= 2 they are even)
  const bool wide_pref = layout == TPDQ_LAYOUT_TILED && meta == kMetaGroup && !gated &&
                         (int64_t)K * N >= kWideMinWeights && M >= 3;
  const bool small_m = meta != kMetaGroup || M <= 4;
  const bool fits = meta_bytes + x_bytes <= budget && small_m && !wide_pref;
  int am;
  if (operand == kOperandGather) {
    // the gather inside the kernel loads the permutation (K x 4 bytes) and X
    // in every 16-column workgroup: on grids of more than kGatherOnceTiles
    // tiles the caller gathers X' once instead
    if (meta_bytes + x_bytes + xr_bytes > budget || meta != kMetaGroup || M > 4 || wide_pref ||
        ntiles > kGatherOnceTiles)
      return false;
    am = kALdsGather;
  } else if (operand == kOperandPrepared) {
    am = kAGlobalPrep;
  } else {
    am = fits ? kALds : kAGlobal;
  }
  if (a_global(am) && mt > 1 && nw > 8) nw = 8;
  int tn = 1;
  if (meta == kMetaGroup) {
    // the ordered kernel streams best with 8 waves (about 8 blocks of 128
    // rows each) when the grid has no more workgroups than CUs, else with 4
    // (measured on the Llama-70B and Granite-20B shapes); with X read from
    // global memory, 4 waves, and two tiles per workgroup (half the re-reads
    // of X) from 384 tiles on: Granite-20B TP=4 at M = 16 (384 tiles, 192
    // workgroups) 14.7 -> 9.7 us per GEMM, while the Llama-70B TP=8 GEMM1
    // (224 tiles) is slower paired (10.5 -> 11.1 us)
    const int nblk = (K + 127) / 128;
    nw = (!a_global(am) && nblk >= 48 && ntiles <= 256) ? 8 : 4;
    if (a_global(am) && ntiles >= 384) tn = 2;
  }
  if (gated) tn = 2;  // the gate and up streams of one 16-column tile
  // two weight streams over two or four row tiles: 8 waves (two per SIMD)
  // leave too few registers (the compiler spills), so 4
  if (gated && mt >= 2) nw = 4;
  // the wide kernel when X is read from global memory and the weights are
  // large (the decode kernel re-reads X for every 16 columns): 8 waves over
  // 128 columns share X through LDS, K split until about kWideTargetWgs
  // workgroups stream
  p->wide = !gated && meta == kMetaGroup && layout == TPDQ_LAYOUT_TILED && a_global(am) &&
            ((int64_t)K * N >= kWideMinWeights ||
             (am == kAGlobal && (mt == 4 || (mt == 2 && K >= N)) &&
              (int64_t)K * N >= kWideMinWeightsRowMajor));
  p->ks = 1;
  if (p->wide) {
    const int nblk = (K + 127) / 128;
    const int wgs = (ntiles + kWideWaves - 1) / kWideWaves;
    p->ks = std::max(1, std::min((kWideTargetWgs + wgs - 1) / wgs, std::max(1, nblk / 4)));
  }
  p->tn = tn;
  p->gated = gated;
  p->dt = dt;
  p->layout = layout;
  p->meta = meta;
  p->amode = am;
  p->nw = nw;
  p->mt = mt;
  p->spg = spg;
  p->meta_rows = meta_rows;
  p->lds_x_off = (int)meta_bytes;
  p->lds_xr_off = (int)(meta_bytes + x_bytes);
  size_t need = a_global(am) ? meta_bytes : meta_bytes + x_bytes;  // <= budget when staged
  if (am == kALdsGather) need += xr_bytes;
  const size_t red_final = (size_t)nw * mt * tn * 1024;  // reduce_store's partial tiles
  if (need < red_final) need = red_final;
  p->lds_bytes = need;
  if (p->wide) {
    p->lds_bytes = (size_t)2 * mt * 16 * 1024;  // two chunks of 4 blocks of activations
    return decode_kernel(*p) != nullptr;
  }
  return decode_kernel(*p) != nullptr;
}

hipError_t launch_decode(const GemmArgs& a0, const DecodePlan& p, float* part, hipStream_t s) {
  if (p.wide) {
    DecodeKernel k = decode_kernel(p);
    if (!k || (p.ks > 1 && !part)) return hipErrorInvalidValue;
    GemmArgs a = a0;
    a.ks = p.ks;
    a.part = part;
    hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_bytes);
    if (e != hipSuccess) return e;
    const int ntiles = (a.N + kTileN - 1) / kTileN;
    const int wgs = (ntiles + kWideWaves - 1) / kWideWaves;
    hipLaunchKernelGGL(k, dim3(wgs * p.ks), dim3(kWideWaves * 64), p.lds_bytes, s, a);
    e = hipGetLastError();
    if (e != hipSuccess || p.ks == 1) return e;
    return launch_splitk_reduce(part, p.ks, a.M, a.N, a.Y, a.ldy, p.dt, s);
  }
  DecodeKernel k = decode_kernel(p);
  if (!k) return hipErrorInvalidValue;
  GemmArgs a = a0;
  a.meta_rows = p.meta_rows;
  a.lds_x_off = p.lds_x_off;
  a.lds_xr_off = p.lds_xr_off;
  if (p.lds_bytes > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)kLdsMax);
    if (e != hipSuccess) return e;
  }
  const int ntiles = (a.N + kTileN - 1) / kTileN;
  const int grid = p.gated ? ntiles : (ntiles + p.tn - 1) / p.tn;  // gated: both streams, one tile
  hipLaunchKernelGGL(k, dim3(grid), dim3(p.nw * 64), p.lds_bytes, s, a);
  return hipGetLastError();
}

hipError_t launch_gather_plain(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                               uint16_t* Xp, hipStream_t s) {
  const int64_t total = (int64_t)M * (K >> 3);
  int blocks = (int)((total + 63) / 64);
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_gather_plain, dim3(blocks), dim3(64), 0, s, X, ldx, M, K, perm, Xp);
  return hipGetLastError();
}

hipError_t launch_gather_prep(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                              int layout, uint16_t* Xp, hipStream_t s) {
  const int64_t total = (int64_t)((M + kTileM - 1) / kTileM) * 4 * ((K + 127) / 128) * 64;
  // one record per thread, 64-thread workgroups: the work is a few hundred
  // KiB of dependent loads, so it is spread over as many CUs as it fills
  int blocks = (int)((total + 63) / 64);
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_gather_prep, dim3(blocks), dim3(64), 0, s, X, ldx, M, K, perm,
                     layout == TPDQ_LAYOUT_TILED ? 1 : 0, Xp);
  return hipGetLastError();
}

}  // namespace tpdq
