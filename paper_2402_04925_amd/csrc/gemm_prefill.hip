// W4A16 dequantize-and-multiply for prefill-sized batches on gfx950: sorted
// rows (the ordered path of Alg. 3, group of row k = k / G), tiled weights.
//
// At M in the thousands the product is a dense contraction and the MFMA pipe
// bounds it (2 M K N flops against K N / 2 bytes of weights), so the kernel
// is a register-blocked MFMA GEMM:
//   * a workgroup of 8 waves (two per SIMD, so that one wave's waits are
//     covered by the other's MFMAs) computes a 128 x 512 tile of Y; each wave
//     owns 64 columns over all 128 rows (8 row tiles x 4 column tiles of
//     v_mfma_f32_16x16x32_f16), so that each dequantized weight fragment
//     feeds 8 MFMAs and the unpack and scaling cost about 2 VALU per MFMA;
//   * K advances one 128-row block at a time (4 MFMA steps of 32 rows);
//   * every operand goes from global memory straight to LDS (buffer loads
//     with the LDS bit, one record of 64 lanes per instruction): activations
//     laid out as the A operand, the wave's weights as they are tiled (one
//     16-byte record per lane and 16-column tile: the B operand), the scales
//     and zeros of the wave's columns; nothing is staged through registers,
//     so the loop keeps one copy of the accumulators;
//   * two stages: block b + 1 is loaded while block b is multiplied, its
//     loads issued one after each column tile's MFMAs (a burst of them at
//     the start of a block stalls the issuing waves); one barrier per block
//     hands a stage from its loads to its readers and back.
// The waits are explicit: before block b each wave waits for its own loads
// of block b (the most recent ones), and the barrier then makes every wave's
// LDS writes visible.
// Dequantizing to fp16 before the MFMA rounds each weight once (relative
// error 2^-12); the decode kernels keep q - z exact and scale in fp32, but
// here that would double the accumulator registers and the VALU work per
// MFMA. With bf16 activations the weight is formed in fp32 and rounded once
// to bf16 (relative error 2^-9), about four times the VALU work of fp16.
#include "kernels_common.h"

#include <algorithm>

namespace tpdq {
namespace {

constexpr int kPWT = 4;    // column tiles per wave
constexpr int kPWwave = kPWT * 64 * 16;
constexpr int kPMwave = 3 * 256;
// LDS per stage with RT row tiles and NW waves: activations
// [RT row tiles][4 steps][64 lanes] x 16 B, then per wave its weights
// [4 tiles][64 lanes] x 16 B and its metadata (three 256-byte records)
__host__ __device__ constexpr int pf_stage(int rt, int nw) {
  return rt * 4 * 64 * 16 + nw * (kPWwave + kPMwave);
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

template <int BYTES>
__device__ __forceinline__ void dma_to_lds(__amdgpu_buffer_rsrc_t r, void* dst, uint32_t off) {
  static_assert(BYTES == 4 || BYTES == 16, "4- or 16-byte records");
  if constexpr (BYTES == 16)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)dst, 16, off, 0, 0, 0);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)dst, 4, off, 0, 0, 0);
}

__device__ __forceinline__ u4_t dequant_scaled(const UnpackConsts<kF16>& kc, uint32_t w, uint32_t z1024,
                                               uint32_t z64, uint32_t s2) {
  const h8_t d = unpack_sub(kc, w, z1024, z64);
  const h2_t s = as_h2(s2);
  const h8_t sv = {s.x, s.y, s.x, s.y, s.x, s.y, s.x, s.y};
  return __builtin_bit_cast(u4_t, d * sv);
}

// bf16: s (q - z) = (128 + q) s - (128 + z) s with zs = (128 + z) s; both
// products are exact in fp32 (8 significant bits each), so one FMA gives
// s (q - z) exactly and the conversion rounds it once.
__device__ __forceinline__ u4_t dequant_scaled_bf16(const UnpackConsts<kBF16>& kc, uint32_t w,
                                                    float s, float zs) {
  const u4_t b = unpack_bias_bf16(kc, w);
  u4_t r;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    r[i] = pack2<kBF16>(__builtin_fmaf(as_f32(b[i] << 16), s, -zs),
                        __builtin_fmaf(as_f32(b[i] & 0xFFFF0000u), s, -zs));
  return r;
}

// RT row tiles (16 RT rows of Y per workgroup), NW waves (64 columns each),
// ST stages (2 or 3) of LDS. With a.ks > 1 the workgroup covers one of ks
// contiguous ranges of 128-row blocks of K and writes its fp32 partial tile
// to a.part[split][M][N] (k_splitk_reduce sums the splits); else it writes
// fp16 Y.
// Two waves per SIMD (the 8-wave workgroup, or two 4-wave workgroups per CU):
// 256 registers per lane, with the accumulators in the architectural VGPRs
// (no accumulator copies between loop iterations).
template <int SPG, int NW, int ST, int RT, int DT>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2))) void k_prefill(GemmArgs a) {
  // groups per 128-row block: G = 32, 64, 128 -> 4, 2, 1; G = 256 -> one
  // group spans two blocks (each block loads it)
  constexpr int GPK = SPG >= 4 ? 1 : 4 / SPG;
  constexpr int NSD = (GPK + 1) / 2;  // scale records per wave and block
  static_assert((RT * 4) % NW == 0, "activation records split evenly over the waves");
  constexpr int AREC = RT * 4 / NW;   // activation records per wave and block
  // loads per wave and block: activations, scales, zeros, weights
  constexpr int LPB = AREC + NSD + 1 + kPWT;
  constexpr int STAGE = pf_stage(RT, NW);
  constexpr int ABYTES = RT * 4 * 64 * 16;
  constexpr int BM = 16 * RT;
  constexpr int BN = 64 * NW;
  extern __shared__ __align__(16) unsigned char smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int nbm = (a.M + BM - 1) / BM;
  const int ks = a.ks > 1 ? a.ks : 1;
  const int ntl = (int)(gridDim.x / ks);  // output tiles
  // consecutive workgroups (one XCD) take neighbouring tiles of one split:
  // they share its activations in L2
  const int lt = xcd_tile(blockIdx.x, gridDim.x);
  const int kidx = lt / ntl;
  const int tl = lt - kidx * ntl;
  const int bn = tl / nbm;
  const int bm = tl - bn * nbm;
  const int row0 = bm * BM;
  const int col0 = bn * BN;
  const int cw = col0 + 64 * wave;
  const int nblk_all = (a.K + 127) >> 7;
  // this workgroup's blocks [kb0, kb1)
  const int kb0 = (int)((int64_t)nblk_all * kidx / ks);
  const int kb1 = (int)((int64_t)nblk_all * (kidx + 1) / ks);
  const int ng = a.num_groups;
  const int ntiles = (a.N + kTileN - 1) / kTileN;
  const UnpackConsts<DT> kc;

  // sources: rows past M, groups past the last one and tiles past N load
  // zeros from the resource bounds
  // per-lane parts of the offsets
  // activations: record (rt, u) of block b, lane l = row 16 rt + l % 16,
  // columns 128 b + 32 u + 8 (l / 16) .. +7
  const uint32_t x_lane = ((uint32_t)j * (uint32_t)a.ldx + 8u * (uint32_t)kq) * 2u;
  const uint32_t x_rt = 16u * (uint32_t)a.ldx * 2u;
  // scales: record d, lane l = group 2 d + l / 32, columns 2 (l % 32), +1
  const uint32_t s_lane = (uint32_t)(lane >> 5) * (uint32_t)a.lds * 2u +
                          ((uint32_t)cw + 2u * (uint32_t)(lane & 31)) * 2u;
  const uint32_t z_lane =
      ((uint32_t)(lane >> 3) * (uint32_t)a.ldz + (uint32_t)(cw >> 3) + (uint32_t)(lane & 7)) * 4u;
  // zeros: lane l = group l / 8, word l % 8 of the wave's 8
  const bool z_used = (lane >> 3) < GPK;
  // weights: tile (cw / 16 + i), block b: lane l's 16 bytes
  const uint32_t w_lane = ((uint32_t)(cw >> 4) * (uint32_t)a.ldq + 4u * (uint32_t)lane) * 4u;
  const uint32_t w_tile = (uint32_t)a.ldq * 4u;

  // per-lane offsets inside one block's window of each source, the same for
  // every block; the window (a buffer resource: base and size in scalar
  // registers) moves with the block, so a load needs no per-block vector
  // arithmetic. Blocks past the workgroup's range get an empty window: their
  // loads return zeros and cost no traffic.
  const int bl = nblk_all - 1;
  uint32_t offA[AREC], offAt[AREC], offS[NSD], offW[kPWT];
#pragma unroll
  for (int k = 0; k < AREC; ++k) {
    const int rec = AREC * wave + k, rt = rec >> 2, u = rec & 3;
    offA[k] = x_lane + (uint32_t)rt * x_rt + (uint32_t)(32 * u) * 2u;
    // the last block: the lane's octet loads zeros past K (the padding of X
    // past K is never read)
    offAt[k] = 128 * bl + 32 * u + 8 * kq < a.K ? offA[k] : kOutOfRange;
  }
#pragma unroll
  for (int d = 0; d < NSD; ++d)
    offS[d] = 2 * d + (lane >> 5) < GPK ? s_lane + (uint32_t)(2 * d) * (uint32_t)a.lds * 2u : kOutOfRange;
  const uint32_t offZ = z_used ? z_lane : kOutOfRange;
#pragma unroll
  for (int i = 0; i < kPWT; ++i) offW[i] = w_lane + (uint32_t)i * w_tile;
  const uint32_t xbytes = (uint32_t)(a.M - row0) * (uint32_t)a.ldx * 2u;
  const uint32_t wbytes = (uint32_t)ntiles * (uint32_t)a.ldq * 4u;

  // load k (0 <= k < LPB) of block b into LDS stage st; each item is exactly
  // one load (the wait counts rely on it)
  auto dma_item = [&](int b, int st, int k) {
    unsigned char* sb = smem + st * STAGE;
    unsigned char* wb = sb + ABYTES + wave * (kPWwave + kPMwave);
    unsigned char* mb = wb + kPWwave;
    const int g0 = (128 * b) / (32 * SPG);
    const bool bok = b < kb1;
    if (k < AREC) {
      const int rec = AREC * wave + k;
      const __amdgpu_buffer_rsrc_t r = buffer_rsrc(a.X + (int64_t)row0 * a.ldx + 128 * b,
                                                   bok ? xbytes - 256u * (uint32_t)b : 0u);
      dma_to_lds<16>(r, sb + rec * 1024, b == bl ? offAt[k] : offA[k]);
    } else if (k < AREC + NSD) {
      const int d = k - AREC;
      const __amdgpu_buffer_rsrc_t r = buffer_rsrc(a.sc + (int64_t)g0 * a.lds,
                                                   bok ? (uint32_t)(ng - g0) * (uint32_t)a.lds * 2u : 0u);
      dma_to_lds<4>(r, mb + d * 256, offS[d]);
    } else if (k == AREC + NSD) {
      const __amdgpu_buffer_rsrc_t r = buffer_rsrc(a.qz + (int64_t)g0 * a.ldz,
                                                   bok ? (uint32_t)(ng - g0) * (uint32_t)a.ldz * 4u : 0u);
      dma_to_lds<4>(r, mb + 512, offZ);
    } else {
      const int i = k - AREC - NSD - 1;
      const __amdgpu_buffer_rsrc_t r = buffer_rsrc(a.qw + (int64_t)256 * b,
                                                   bok ? wbytes - 1024u * (uint32_t)b : 0u);
      dma_to_lds<16>(r, wb + i * 1024, offW[i]);
    }
  };
  auto issue = [&](int b, int st) {
#pragma unroll
    for (int k = 0; k < LPB; ++k) dma_item(b, st, k);
  };

  f4_t acc[RT][kPWT];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int i = 0; i < kPWT; ++i) acc[r][i] = f4_t{0.f, 0.f, 0.f, 0.f};

  // block in stage st; the loads of block bn go out one after each column
  // tile's MFMAs, into stage sn
  auto compute = [&](int st, int bnext, int sn) {
    const u4_t* ab = (const u4_t*)(smem + st * STAGE);
    const u4_t* wb = (const u4_t*)(smem + st * STAGE + ABYTES + wave * (kPWwave + kPMwave));
    const unsigned char* mb = (const unsigned char*)wb + kPWwave;
    u4_t w[kPWT];
#pragma unroll
    for (int i = 0; i < kPWT; ++i) w[i] = wb[i * 64 + lane];
    uint32_t z1024[kPWT], z64[kPWT], s2[kPWT];
    float sf[kPWT], zs[kPWT];  // bf16
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool open = SPG >= 4 ? u == 0 : (u % SPG) == 0;
      if (open) {
        const int gi = SPG >= 4 ? 0 : u / SPG;
#pragma unroll
        for (int i = 0; i < kPWT; ++i) {
          const int c = 16 * i + j;
          const uint32_t sv = *(const uint16_t*)(mb + gi * 128 + 2 * c);
          const uint32_t zw = *(const uint32_t*)(mb + 512 + gi * 32 + 4 * (c >> 3));
          const uint32_t zc = ((zw >> (4 * (c & 7))) & 0xFu) + (uint32_t)a.zoff;  // up to 16
          if constexpr (DT == kBF16) {
            sf[i] = bits_to_float<kBF16>(sv);
            zs[i] = (128.f + (float)zc) * sf[i];
          } else {
            z1024[i] = (0x6400u | zc) * 0x10001u;
            z64[i] = (0x5400u | (zc << 4)) * 0x10001u;
            s2[i] = sv * 0x10001u;
          }
        }
      }
      u4_t av[RT];
#pragma unroll
      for (int r = 0; r < RT; ++r) av[r] = ab[(r * 4 + u) * 64 + lane];
#pragma unroll
      for (int i = 0; i < kPWT; ++i) {
        u4_t bv;
        if constexpr (DT == kBF16)
          bv = dequant_scaled_bf16(kc, w[i][u], sf[i], zs[i]);
        else
          bv = dequant_scaled(kc, w[i][u], z1024[i], z64[i], s2[i]);
#pragma unroll
        for (int r = 0; r < RT; ++r) acc[r][i] = mfma_k32<DT>(av[r], bv, acc[r][i]);
        if (4 * u + i < LPB) dma_item(bnext, sn, 4 * u + i);
      }
    }
  };

  // Before block b: this wave's loads of block b have landed (with three
  // stages, those of block b + 1 may still be in flight) and its LDS reads of
  // block b - 1 are done; the barrier then publishes every wave's block b
  // and frees the stage that receives the next block.
  auto sync = [&]() {
    if constexpr (ST == 3)
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"(LPB) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };
#pragma unroll
  for (int p = 0; p < ST - 1; ++p) issue(kb0 + p, p);
  int st = 0;
#pragma unroll 1
  for (int b = kb0; b < kb1; ++b) {
    sync();
    const int sn = st == 0 ? ST - 1 : st - 1;
    compute(st, b + ST - 1, sn);
    st = st == ST - 1 ? 0 : st + 1;
  }
  // the loads past the last block (zeros) still write LDS: let them land
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // epilogue: acc[r][i] of lane (j, kq) holds rows 4 kq .. +3 of row tile r,
  // column j of the wave's tile i
  float* part = a.part + (size_t)kidx * a.M * a.N;
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int i = 0; i < kPWT; ++i) {
      const int c = cw + 16 * i + j;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = row0 + 16 * r + 4 * kq + e;
        if (row < a.M && c < a.N) {
          if (ks > 1)
            part[(int64_t)row * a.N + c] = acc[r][i][e];
          else
            a.Y[(int64_t)row * a.ldy + c] = float_to_bits<DT>(acc[r][i][e]);
        }
      }
    }
}

// Y[m][n] = round(sum over s of part[s][m][n]) to the element type, the splits added in order s =
// 0, 1, ... (the result does not depend on which split finished first). Four
// columns per thread: one 16-byte load per split, one 8-byte store (N % 4 ==
// 0 and 16-byte aligned rows; otherwise one column per thread).
template <int DT>
__global__ __launch_bounds__(256) void k_splitk_reduce(const float* __restrict__ part, int ks, int M,
                                                       int N, uint16_t* __restrict__ Y, int64_t ldy) {
  const int64_t plane = (int64_t)M * N;
  if ((N & 3) == 0 && (ldy & 3) == 0) {
    const int n4 = N >> 2;
    const int64_t total = (int64_t)M * n4;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
      const int m = (int)(i / n4);
      const int c0 = (int)(i - (int64_t)m * n4) * 4;
      const float* src = part + (int64_t)m * N + c0;
      f4_t v = *(const f4_t*)src;
      for (int s = 1; s < ks; ++s) v += *(const f4_t*)(src + s * plane);
      const uint32_t lo = pack2<DT>(v[0], v[1]);
      const uint32_t hi = pack2<DT>(v[2], v[3]);
      *(uint2*)(Y + (int64_t)m * ldy + c0) = make_uint2(lo, hi);
    }
    return;
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < plane;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(i / N);
    const int c = (int)(i - (int64_t)m * N);
    float v = part[i];
    for (int s = 1; s < ks; ++s) v += part[s * plane + i];
    Y[(int64_t)m * ldy + c] = float_to_bits<DT>(v);
  }
}

__global__ __launch_bounds__(256) void k_gather_rows(const uint16_t* __restrict__ X, int64_t ldx,
                                                     int K, const int32_t* __restrict__ perm,
                                                     uint16_t* __restrict__ Xp) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint16_t* xl = (uint16_t*)smem;
  const int m = blockIdx.x;
  const uint16_t* xr = X + (int64_t)m * ldx;
  const int kw = K >> 3;
  for (int o = threadIdx.x; o < kw; o += blockDim.x) *(u4_t*)(xl + 8 * o) = *(const u4_t*)(xr + 8 * o);
  __syncthreads();
  const uint32_t kmax = (uint32_t)(K - 1);
  for (int o = threadIdx.x; o < kw; o += blockDim.x) {
    const u4_t p0 = *(const u4_t*)(perm + 8 * o);
    const u4_t p1 = *(const u4_t*)(perm + 8 * o + 4);
    uint32_t x[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = xl[min(p0[e], kmax)];
      x[e + 4] = xl[min(p1[e], kmax)];
    }
    *(u4_t*)(Xp + (int64_t)m * K + 8 * o) =
        u4_t{x[0] | (x[1] << 16), x[2] | (x[3] << 16), x[4] | (x[5] << 16), x[6] | (x[7] << 16)};
  }
}

}  // namespace

bool plan_mtile(int M, int64_t ldx, const tpdq_w4* w, int meta, MtilePlan* p) {
  if (meta != kMetaGroup || w->layout != TPDQ_LAYOUT_TILED) return false;
  const int K = w->K, N = w->N, G = w->group_size;
  if (M < kMtileMinM || K % 8 != 0 || G <= 0 || G % 32 != 0) return false;
  const int spg = G / 32;
  if (!(spg == 1 || spg == 2 || spg == 4 || spg == 8)) return false;
  // activation rows on 16 bytes, scale rows on 4 (the LDS loads move 16 and
  // 4 bytes per lane)
  if (ldx % 8 != 0 || w->ld_s % 2 != 0 || ((uintptr_t)w->scales & 3) != 0) return false;
  // byte offsets of the buffer loads are 32-bit
  const int64_t lim = (int64_t)1 << 31;
  const int64_t ntiles = (N + kTileN - 1) / kTileN;
  if (!(ntiles * w->ld_q * 4 < lim && (int64_t)M * ldx * 2 < lim &&
        (int64_t)w->num_groups * w->ld_s * 2 < lim && (int64_t)w->num_groups * w->ld_z * 4 < lim))
    return false;
  MtilePlan q{};
  if (M >= kPrefillMinM) {
    // a dense contraction: 8 waves (two per SIMD) over 128 x 512 tiles
    q.rt = 8;
    q.nw = 8;
    q.st = 2;
    q.ks = 1;
  } else {
    // below prefill sizes the weight stream bounds the product; worth it
    // only when the weights are large enough that the decode kernels'
    // per-workgroup re-reads of X dominate: 64 x 512 tiles, 8 waves (two per
    // SIMD, one workgroup per CU), K split as far as the workgroups still
    // fit the kMtileSlots CUs in one round. Llama-70B TP=1 at M = 64 (MLP):
    // 109.5 us with 64 x 256 tiles of 4 waves in 512 slots (two per CU),
    // 106.3 us here (GEMM2 52.4 -> 48.9 us: 8 waves share one copy of the
    // activations); more splits than fit one round are slower (8 waves in
    // 320 slots: GEMM1 280 workgroups, 144 us), and so is one wave per SIMD
    if ((int64_t)K * N < kMtileMinWeights) return false;
    q.rt = 4;
    q.nw = 8;
    q.st = 2;
    const int nblk = (K + 127) / 128;
    const int tiles = ((M + 63) / 64) * ((N + 511) / 512);
    int ks = kMtileSlots / tiles;
    ks = std::max(1, std::min(ks, nblk / 4));
    if ((int64_t)ks * M * N * 4 >= lim) ks = 1;
    q.ks = ks;
  }
  *p = q;
  return true;
}

size_t mtile_part_bytes(const MtilePlan& p, int M, int N) {
  return p.ks > 1 ? align_up((size_t)p.ks * M * N * 4) : 0;
}

template <int NW, int ST, int RT, int DT>
hipError_t launch_mtile_t(const GemmArgs& a, int ks, hipStream_t s) {
  typedef void (*Kern)(GemmArgs);
  Kern k = nullptr;
  switch (a.G / 32) {
    case 1: k = k_prefill<1, NW, ST, RT, DT>; break;
    case 2: k = k_prefill<2, NW, ST, RT, DT>; break;
    case 4: k = k_prefill<4, NW, ST, RT, DT>; break;
    case 8: k = k_prefill<8, NW, ST, RT, DT>; break;
  }
  if (!k) return hipErrorInvalidValue;
  const int lds = ST * pf_stage(RT, NW);
  hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  const int grid = ((a.M + 16 * RT - 1) / (16 * RT)) * ((a.N + 64 * NW - 1) / (64 * NW)) * ks;
  hipLaunchKernelGGL(k, dim3(grid), dim3(NW * 64), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_mtile(const GemmArgs& a0, const MtilePlan& p, float* part, hipStream_t s) {
  GemmArgs a = a0;
  a.ks = p.ks;
  a.part = part;
  if (p.ks > 1 && !part) return hipErrorInvalidValue;
  hipError_t e;
  const bool bf = a.dt == kBF16;
  if (p.rt == 8 && p.nw == 8 && p.st == 2)
    e = bf ? launch_mtile_t<8, 2, 8, kBF16>(a, p.ks, s) : launch_mtile_t<8, 2, 8, kF16>(a, p.ks, s);
  else if (p.rt == 4 && p.nw == 8 && p.st == 2)
    e = bf ? launch_mtile_t<8, 2, 4, kBF16>(a, p.ks, s) : launch_mtile_t<8, 2, 4, kF16>(a, p.ks, s);
  else
    return hipErrorInvalidValue;
  if (e != hipSuccess || p.ks == 1) return e;
  return launch_splitk_reduce(part, p.ks, a.M, a.N, a.Y, a.ldy, a.dt, s);
}

hipError_t launch_splitk_reduce(const float* part, int ks, int M, int N, uint16_t* Y, int64_t ldy,
                                int dt, hipStream_t s) {
  const int64_t total = (int64_t)M * N / 4 + 1;
  const int blocks = (int)std::min<int64_t>((total + 255) / 256, 16384);
  if (dt == kBF16)
    hipLaunchKernelGGL(k_splitk_reduce<kBF16>, dim3(blocks), dim3(256), 0, s, part, ks, M, N, Y, ldy);
  else
    hipLaunchKernelGGL(k_splitk_reduce<kF16>, dim3(blocks), dim3(256), 0, s, part, ks, M, N, Y, ldy);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                              uint16_t* Xp, hipStream_t s) {
  const size_t lds = (size_t)K * 2;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k_gather_rows,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_gather_rows, dim3(M), dim3(256), lds, s, X, ldx, K, perm, Xp);
  return hipGetLastError();
}

}  // namespace tpdq
