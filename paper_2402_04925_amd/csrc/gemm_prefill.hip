// W4A16 dequantize-and-multiply for prefill-sized batches on gfx950: sorted
// rows (the ordered path of Alg. 3, group of row k = k / G), tiled weights.
//
// At M in the thousands the product is a dense contraction and the MFMA pipe
// bounds it (2 M K N flops against K N / 2 bytes of weights), so the kernel
// is a classic register-blocked MFMA GEMM:
//   * a workgroup computes a 128 x 256 tile of Y with 8 waves, each a 64 x 64
//     sub-tile (4 row tiles x 4 column tiles of v_mfma_f32_16x16x32_f16), so
//     that two waves share each SIMD and hide each other's load latency;
//   * K advances one 128-row block at a time (4 MFMA steps of 32 rows);
//   * the activations of the block (128 rows x 128 columns, fp16) are staged
//     in LDS in MFMA operand order, double-buffered so that the next block's
//     loads overlap the current block's MFMAs;
//   * the weights go straight from the tiled layout to registers (one 16-byte
//     load per lane per 16-column tile and block), are unpacked to exact
//     q - z and scaled to fp16 (s (q - z)) right before the MFMA; one
//     (scale, zero) per column and group comes from LDS, staged with the
//     activations.
// Dequantizing to fp16 before the MFMA rounds each weight once (relative
// error 2^-12); the decode kernels keep q - z exact and scale in fp32, but
// here that would double the accumulator registers and the VALU work per
// MFMA.
#include "kernels_common.h"

namespace tpdq {
namespace {

constexpr int kPBM = 128;  // rows of Y per workgroup
constexpr int kPBN = 256;  // columns of Y per workgroup (16 tiles of 16)
constexpr int kPNW = 8;    // waves: 2 (rows) x 4 (columns)
constexpr int kPWT = 4;    // column tiles per wave
constexpr int kPNT = kPNW * 64;
// LDS: two activation buffers [8 row tiles][4 steps][64 lanes] x 16 B and
// two metadata buffers [4 groups][256 columns] x 4 B
constexpr int kPAbuf = 8 * 4 * 64 * 16;
constexpr int kPMbuf = 4 * kPBN * 4;
constexpr int kPLds = 2 * kPAbuf + 2 * kPMbuf;

// fp16 x2 of the dequantized weights: (q - z) * s
__device__ __forceinline__ h8_t dequant_scaled(const UnpackConsts& kc, uint32_t w, uint32_t z1024,
                                               uint32_t z64, uint32_t s2) {
  const h8_t d = unpack_sub(kc, w, z1024, z64);
  const h2_t s = as_h2(s2);
  const h8_t sv = {s.x, s.y, s.x, s.y, s.x, s.y, s.x, s.y};
  return d * sv;
}

template <int SPG>
__global__ __launch_bounds__(kPNT) void k_prefill(GemmArgs a) {
  // groups per 128-row block: G = 32, 64, 128 -> 4, 2, 1; G = 256 -> one
  // group spans two blocks
  constexpr int GPK = SPG >= 4 ? 1 : 4 / SPG;
  extern __shared__ __align__(16) unsigned char smem[];
  u4_t* abuf[2] = {(u4_t*)smem, (u4_t*)(smem + kPAbuf)};
  uint32_t* mbuf[2] = {(uint32_t*)(smem + 2 * kPAbuf), (uint32_t*)(smem + 2 * kPAbuf + kPMbuf)};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int wm = wave & 1, wn = wave >> 1;
  const int nbn = (a.N + kPBN - 1) / kPBN;
  const int bm = blockIdx.x / nbn;
  const int bn = blockIdx.x - bm * nbn;
  const int row0 = bm * kPBM;
  const int col0 = bn * kPBN;
  const int kw = a.K >> 3;
  const int nblk = (a.K + 127) >> 7;
  const int ng = a.num_groups;
  const int ntiles = (a.N + kTileN - 1) / kTileN;
  const UnpackConsts kc;

  // sources (buffer resources: rows past M, columns past N and octets past K
  // load zeros)
  const __amdgpu_buffer_rsrc_t rx = buffer_rsrc(a.X, (uint32_t)a.M * (uint32_t)a.ldx * 2u);
  const __amdgpu_buffer_rsrc_t rw =
      buffer_rsrc(a.qw, (uint32_t)ntiles * (uint32_t)a.ldq * 4u);
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(a.sc, (uint32_t)ng * (uint32_t)a.lds * 2u);
  const __amdgpu_buffer_rsrc_t rz = buffer_rsrc(a.qz, (uint32_t)ng * (uint32_t)a.ldz * 4u);

  // activation piece p (0..3) of this thread: row tid / 16 + 32 p of the
  // tile, octet tid % 16 of the block
  constexpr int AP = kPBM * 16 / kPNT;
  const int a_oct = tid & 15;
  auto load_a = [&](int b, u4_t (&x)[AP]) {
    const int o = 16 * b + a_oct;
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      const int r = row0 + (tid >> 4) + (kPNT / 16) * p;
      const uint32_t off = (r < a.M && o < kw) ? ((uint32_t)r * (uint32_t)a.ldx + (uint32_t)o * 8u) * 2u
                                               : kOutOfRange;
      x[p] = buffer_load16(rx, off);
    }
  };
  auto store_a = [&](u4_t* dst, const u4_t (&x)[AP]) {
    // record [row tile][step][lane]: lane = 16 (octet % 4) + row % 16
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      const int r = (tid >> 4) + (kPNT / 16) * p;
      dst[((r >> 4) * 4 + (a_oct >> 2)) * 64 + (a_oct & 3) * 16 + (r & 15)] = permute_octet(x[p]);
    }
  };
  // metadata of the groups of block b for column col0 + tid
  // (threads tid < 256: one column each)
  auto load_m = [&](int b, uint32_t (&sv)[GPK], uint32_t (&zv)[GPK]) {
    const int c = col0 + tid;
    const int gb = (4 * b) / SPG;
#pragma unroll
    for (int gi = 0; gi < GPK; ++gi) {
      const int g = gb + gi;
      const bool ok = tid < kPBN && c < a.N && g < ng;
      sv[gi] = buffer_load2(rs, ok ? ((uint32_t)g * (uint32_t)a.lds + (uint32_t)c) * 2u : kOutOfRange);
      zv[gi] = buffer_load4(rz, ok ? ((uint32_t)g * (uint32_t)a.ldz + (uint32_t)(c >> 3)) * 4u
                                   : kOutOfRange);
    }
  };
  auto store_m = [&](uint32_t* dst, const uint32_t (&sv)[GPK], const uint32_t (&zv)[GPK]) {
    const uint32_t shift = 4u * (uint32_t)((col0 + tid) & 7);
#pragma unroll
    for (int gi = 0; gi < GPK; ++gi)
      if (tid < kPBN) dst[gi * kPBN + tid] = (sv[gi] & 0xFFFFu) | (((zv[gi] >> shift) & 0xFu) << 16);
  };
  // weights of block b for the wave's column tiles
  const int tw0 = col0 / kTileN + wn * kPWT;
  auto load_w = [&](int b, u4_t (&w)[kPWT]) {
#pragma unroll
    for (int i = 0; i < kPWT; ++i) {
      const int t = tw0 + i;
      const uint32_t off = (t < ntiles && b < nblk)
                               ? ((uint32_t)t * (uint32_t)a.ldq + (uint32_t)b * 256u + (uint32_t)lane * 4u) * 4u
                               : kOutOfRange;
      w[i] = buffer_load16<kNonTemporal>(rw, off);
    }
  };

  f4_t acc[4][kPWT];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int i = 0; i < kPWT; ++i) acc[r][i] = f4_t{0.f, 0.f, 0.f, 0.f};

  // one block: 4 steps of 32 rows from LDS buffer `ab`, weights w
  auto compute = [&](int b, const u4_t* ab, const uint32_t* mb, const u4_t (&w)[kPWT]) {
    uint32_t z1024[kPWT], z64[kPWT], s2[kPWT];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool open = SPG >= 4 ? u == 0 : (u % SPG) == 0;
      if (open) {
        const int gi = SPG >= 4 ? 0 : u / SPG;
#pragma unroll
        for (int i = 0; i < kPWT; ++i) {
          const uint32_t m = mb[gi * kPBN + (wn * kPWT + i) * kTileN + j];
          const uint32_t zc = m >> 16;
          z1024[i] = (0x6400u | zc) * 0x10001u;
          z64[i] = (0x5400u | (zc << 4)) * 0x10001u;
          s2[i] = (m & 0xFFFFu) * 0x10001u;
        }
      }
      h8_t av[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) av[r] = as_h8(ab[((wm * 4 + r) * 4 + u) * 64 + lane]);
#pragma unroll
      for (int i = 0; i < kPWT; ++i) {
        const h8_t bv = dequant_scaled(kc, w[i][u], z1024[i], z64[i], s2[i]);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r][i] = mfma16x16x32(av[r], bv, acc[r][i]);
      }
    }
  };

  // prologue: block 0 to LDS buffer 0, its weights to registers
  u4_t wA[kPWT], wB[kPWT];
  {
    u4_t x[AP];
    uint32_t sv[GPK], zv[GPK];
    load_a(0, x);
    load_m(0, sv, zv);
    load_w(0, wA);
    store_a(abuf[0], x);
    store_m(mbuf[0], sv, zv);
    __syncthreads();
  }
  // block b from buffer b % 2 with weights wc; meanwhile block b + 1 is
  // loaded (activations and metadata to the other buffer, weights to wnx)
  auto step = [&](int b, const u4_t (&wc)[kPWT], u4_t (&wnx)[kPWT]) {
    u4_t x[AP];
    uint32_t sv[GPK], zv[GPK];
    const bool more = b + 1 < nblk;
    if (more) {
      load_a(b + 1, x);
      load_m(b + 1, sv, zv);
    }
    load_w(b + 1, wnx);
    __builtin_amdgcn_sched_barrier(0);
    compute(b, abuf[b & 1], mbuf[b & 1], wc);
    if (more) {
      store_a(abuf[(b + 1) & 1], x);
      store_m(mbuf[(b + 1) & 1], sv, zv);
    }
    __syncthreads();
  };
  for (int b = 0; b < nblk; b += 2) {
    step(b, wA, wB);
    if (b + 1 < nblk) step(b + 1, wB, wA);
  }

  // epilogue: acc[r][i] of lane (j, kq) holds rows 4 kq .. +3 of row tile r,
  // column j of tile i
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int i = 0; i < kPWT; ++i) {
      const int c = (tw0 + i) * kTileN + j;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = row0 + (wm * 4 + r) * kTileM + 4 * kq + e;
        if (row < a.M && c < a.N) a.Y[(int64_t)row * a.ldy + c] = float_to_half_bits(acc[r][i][e]);
      }
    }
}

// X'[m][k] = X[m][perm[k]] in row-major order, one workgroup per row: the row
// is copied to LDS and gathered from there.
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

bool prefill_supported(int M, int K, int N, int G, int layout, int meta, int64_t ldq) {
  if (meta != kMetaGroup || layout != TPDQ_LAYOUT_TILED) return false;
  if (M < kPrefillMinM || K % 8 != 0 || G % 32 != 0 || K % G != 0) return false;
  const int spg = G / 32;
  if (!(spg == 1 || spg == 2 || spg == 4 || spg == 8)) return false;
  // byte offsets of the buffer loads are 32-bit
  const int64_t ntiles = (N + kTileN - 1) / kTileN;
  return ntiles * ldq * 4 < ((int64_t)1 << 31);
}

hipError_t launch_prefill(const GemmArgs& a, hipStream_t s) {
  typedef void (*Kern)(GemmArgs);
  Kern k = nullptr;
  switch (a.G / 32) {
    case 1: k = k_prefill<1>; break;
    case 2: k = k_prefill<2>; break;
    case 4: k = k_prefill<4>; break;
    case 8: k = k_prefill<8>; break;
  }
  if (!k) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, kPLds);
  if (e != hipSuccess) return e;
  const int grid = ((a.M + kPBM - 1) / kPBM) * ((a.N + kPBN - 1) / kPBN);
  hipLaunchKernelGGL(k, dim3(grid), dim3(kPNT), kPLds, s, a);
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
