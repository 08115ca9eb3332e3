// W4A16 dequantize-and-multiply for decode-sized batches (M <= 64) on gfx950.
//
// Y[m][n] = sum_k X[m][k] * s[g(k)][n] * (q[k][n] - z[g(k)][n])
// (group quantization of section 1.1; g(k) = g_idx[k] under act-order, Eq. 3,
// or floor(k / G) for sorted rows, Eq. 1 / Alg. 1).
//
// Work decomposition (both kernels):
//   * a workgroup = 4 waves on one 64-column tile; the tile's K range is cut
//     into `splits` workgroups x 4 waves, each wave taking a contiguous run of
//     32-row k-steps (split-K, needed because a decode N gives only 56..448
//     column tiles for 256 CUs);
//   * lane l owns the 4 consecutive columns 4*(l%16)..+3 of the tile and the
//     k octet l/16 of each 32-row step: one 128-bit load of packed int32 words
//     per lane per step, 256 contiguous bytes per octet row of the wave;
//   * the 4 words of a lane feed 4 v_mfma_f32_16x16x32_f16, MFMA c taking the
//     tile's columns c, c+4, c+8, ...; the B operand of a lane is 8 fp16 values
//     of one column over 8 consecutive k, which is exactly one packed word;
//   * the 4 waves' partial tiles are summed in LDS, the `splits` workgroup
//     partials of a tile in the workspace by the last workgroup to arrive
//     (fixed order, so results are bit-reproducible).
//
// Ordered kernel (sorted rows, G % 32 == 0): a 32-row step never straddles a
// group, so each lane loads its group's 4 scales and zeros once per group,
// the MFMAs accumulate sum_k x*(q - z) of the group exactly-scaled in fp32
// (q - z is an exact small integer in fp16), and the scale is applied once per
// group and column: acc += s * group_acc. This is the metadata reuse of Fig. 2.
//
// Row-metadata kernel (act-order, or sorted rows with G % 32 != 0): every one
// of the 8 rows of a lane's octet fetches its own scale and zero through
// g_idx (Fig. 1's naive load) and the weight is dequantized per element to
// fp16 before the MFMA.
#include "tpdq_internal.h"

namespace tpdq {
namespace {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ h2_t as_h2(uint32_t v) { return __builtin_bit_cast(h2_t, v); }
__device__ __forceinline__ uint32_t as_u32(h2_t v) { return __builtin_bit_cast(uint32_t, v); }

__device__ __forceinline__ float half_bits_to_float(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

__device__ __forceinline__ uint16_t float_to_half_bits(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);  // round to nearest even
}

// Workgroups are dispatched round-robin over the 8 XCDs; renumber them so that
// consecutive logical ids (the split-K workgroups of one column tile) share an
// XCD and therefore an L2 for the partial-sum fix-up.
__device__ __forceinline__ int xcd_logical(int b, int nb) {
  if (nb % 8) return b;
  return (b % 8) * (nb / 8) + b / 8;
}

// Packed word -> 8 fp16 values (q - z) of one column, exact.
// OR-ing a nibble into the mantissa of 1024.0 (0x6400) gives 1024 + q; the
// nibbles at bits 4..7 land as 1024 + 16 q and are rescaled by 1/16 inside
// the same fused op. Output order: k0, k4, k1, k5, k2, k6, k3, k7 (the A
// operand is permuted to match, see permute_octet).
__device__ __forceinline__ h8_t unpack_sub(uint32_t w, uint32_t z1024, uint32_t z64) {
  const uint32_t lo = 0x000F000Fu, hi = 0x00F000F0u, magic = 0x64006400u;
  const uint32_t w8 = w >> 8;
  const h2_t inv16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  h2_t b0 = as_h2((w & lo) | magic) - as_h2(z1024);
  h2_t b1 = as_h2((w & hi) | magic) * inv16 - as_h2(z64);
  h2_t b2 = as_h2((w8 & lo) | magic) - as_h2(z1024);
  h2_t b3 = as_h2((w8 & hi) | magic) * inv16 - as_h2(z64);
  h8_t r = {b0.x, b0.y, b1.x, b1.y, b2.x, b2.y, b3.x, b3.y};
  return r;
}

// 8 consecutive fp16 activations x0..x7 -> x0, x4, x1, x5, x2, x6, x3, x7.
__device__ __forceinline__ h8_t permute_octet(u4_t x) {
  u4_t r;
  r.x = (x.x & 0xFFFFu) | (x.z << 16);
  r.y = (x.x >> 16) | (x.z & 0xFFFF0000u);
  r.z = (x.y & 0xFFFFu) | (x.w << 16);
  r.w = (x.y >> 16) | (x.w & 0xFFFF0000u);
  return __builtin_bit_cast(h8_t, r);
}

__device__ __forceinline__ f4_t mfma16x16x32(h8_t a, h8_t b, f4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// LDS reduction of the 4 waves' partial tiles, then either the final fp16
// store (splits == 1) or the split-K partial store and the last-arriver
// fix-up. acc[t][c][e] is row t*16 + 4*(lane/16) + e, column 4*(lane%16) + c.
template <int MT>
__device__ __forceinline__ void finish_tile(const GemmArgs& a, f4_t (&acc)[MT][4], int tile,
                                            int split, float* red) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        red[((wave * MT + t) * 16 + c * 4 + e) * 64 + lane] = acc[t][c][e];
  __syncthreads();

  const bool direct = a.splits == 1;
#pragma unroll
  for (int it = 0; it < MT; ++it) {
    const int item = tid + 256 * it;      // (t, e, lane)
    const int ln = item & 63;
    const int te = item >> 6;
    const int t = te >> 2, e = te & 3;
    const int row = t * kTileM + 4 * (ln >> 4) + e;
    const int colx = tile * kDecodeCols + 4 * (ln & 15);
    float v[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kDecodeWaves; ++w) s += red[((w * MT + t) * 16 + c * 4 + e) * 64 + ln];
      v[c] = s;
    }
    if (row < a.M && colx < a.N) {
      if (direct) {
        u2_t o;
        o.x = (uint32_t)float_to_half_bits(v[0]) | ((uint32_t)float_to_half_bits(v[1]) << 16);
        o.y = (uint32_t)float_to_half_bits(v[2]) | ((uint32_t)float_to_half_bits(v[3]) << 16);
        *(u2_t*)(a.Y + (int64_t)row * a.ldy + colx) = o;
      } else {
        f4_t o = {v[0], v[1], v[2], v[3]};
        *(f4_t*)(a.partials + ((int64_t)split * a.M + row) * a.N + colx) = o;
      }
    }
  }
  if (direct) return;

  // split-K fix-up: the last workgroup of the tile to arrive sums the partials
  // in split order and writes the fp16 tile, then re-arms the counter.
  __shared__ int is_last;
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const uint32_t prev = atomicAdd(a.counters + tile, 1u);
    is_last = (prev == (uint32_t)(a.splits - 1));
  }
  __syncthreads();
  if (!is_last) return;
  __threadfence();
  const int nq = a.M * (kDecodeCols / 4);
  for (int item = tid; item < nq; item += 256) {
    const int row = item >> 4;
    const int colx = tile * kDecodeCols + 4 * (item & 15);
    if (colx >= a.N) continue;
    f4_t s = {0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < a.splits; ++sp)
      s += *(const f4_t*)(a.partials + ((int64_t)sp * a.M + row) * a.N + colx);
    u2_t o;
    o.x = (uint32_t)float_to_half_bits(s.x) | ((uint32_t)float_to_half_bits(s.y) << 16);
    o.y = (uint32_t)float_to_half_bits(s.z) | ((uint32_t)float_to_half_bits(s.w) << 16);
    *(u2_t*)(a.Y + (int64_t)row * a.ldy + colx) = o;
  }
  if (tid == 0) a.counters[tile] = 0u;
}

// ---------------------------------------------------------------------------
// Ordered kernel: sorted rows, group of row k = k / G, G % 32 == 0.
// ---------------------------------------------------------------------------
template <int MT>
__global__ __launch_bounds__(256) void k_decode_ordered(GemmArgs a) {
  __shared__ float red[kDecodeWaves * MT * 16 * 64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int tile = logical / a.splits;
  const int split = logical - tile * a.splits;
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int col = tile * kDecodeCols + 4 * j;
  const bool col_ok = col < a.N;
  const int kw = a.K >> 3;
  const int nks = (a.K + 31) >> 5;
  const int nw = a.splits * kDecodeWaves;
  const int wi = split * kDecodeWaves + wave;
  int ks = (int)((int64_t)nks * wi / nw);
  const int ks_end = (int)((int64_t)nks * (wi + 1) / nw);
  const int steps_per_group = a.G >> 5;

  f4_t acc[MT][4];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[t][c] = f4_t{0.f, 0.f, 0.f, 0.f};

  const uint32_t* qcol = a.qw + col;
  while (ks < ks_end) {
    const int g = ks / steps_per_group;
    const int seg_end = min(ks_end, (g + 1) * steps_per_group);
    float s[4];
    uint32_t z1024[4], z64[4];
    if (col_ok) {
      const u2_t sv = *(const u2_t*)(a.sc + (int64_t)g * a.lds + col);
      const uint32_t zw = a.qz[(int64_t)g * a.ldz + (col >> 3)] >> (4 * (col & 7));
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        s[c] = half_bits_to_float(((c < 2 ? sv.x : sv.y) >> (16 * (c & 1))) & 0xFFFFu);
        const uint32_t zc = (zw >> (4 * c)) & 0xFu;
        z1024[c] = (0x6400u | zc) * 0x10001u;
        z64[c] = (0x5400u | (zc << 4)) * 0x10001u;
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        s[c] = 0.f;
        z1024[c] = 0x64006400u;
        z64[c] = 0x54005400u;
      }
    }
    f4_t gacc[MT][4];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int c = 0; c < 4; ++c) gacc[t][c] = f4_t{0.f, 0.f, 0.f, 0.f};

    for (int k0 = ks; k0 < seg_end; k0 += 4) {
      const int nstep = min(4, seg_end - k0);
      u4_t wv[4];
      h8_t av[4][MT];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int wr = (k0 + u) * 4 + kq;
        const bool ok = u < nstep && wr < kw;
        wv[u] = u4_t{0u, 0u, 0u, 0u};
        if (ok && col_ok) wv[u] = *(const u4_t*)(qcol + (int64_t)wr * a.ldq);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          const int row = t * kTileM + j;
          u4_t xv = u4_t{0u, 0u, 0u, 0u};
          if (ok && row < a.M) xv = *(const u4_t*)(a.X + (int64_t)row * a.ldx + wr * 8);
          av[u][t] = permute_octet(xv);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (u < nstep) {
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const h8_t b = unpack_sub(wv[u][c], z1024[c], z64[c]);
#pragma unroll
            for (int t = 0; t < MT; ++t) gacc[t][c] = mfma16x16x32(av[u][t], b, gacc[t][c]);
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[t][c] += s[c] * gacc[t][c];
    ks = seg_end;
  }
  finish_tile<MT>(a, acc, tile, split, red);
}

// ---------------------------------------------------------------------------
// Row-metadata kernel: each row's scale and zero fetched through its group.
// ACT = true: group = g_idx[k] (clamped into range); false: group = k / G.
// ---------------------------------------------------------------------------
template <int MT, bool ACT>
__global__ __launch_bounds__(256) void k_decode_rowmeta(GemmArgs a) {
  __shared__ float red[kDecodeWaves * MT * 16 * 64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int tile = logical / a.splits;
  const int split = logical - tile * a.splits;
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int col = tile * kDecodeCols + 4 * j;
  const bool col_ok = col < a.N;
  const int kw = a.K >> 3;
  const int nks = (a.K + 31) >> 5;
  const int nw = a.splits * kDecodeWaves;
  const int wi = split * kDecodeWaves + wave;
  const int ks_begin = (int)((int64_t)nks * wi / nw);
  const int ks_end = (int)((int64_t)nks * (wi + 1) / nw);
  const uint32_t gmax = (uint32_t)(a.num_groups - 1);
  const int zshift = 4 * (col & 7);

  f4_t acc[MT][4];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[t][c] = f4_t{0.f, 0.f, 0.f, 0.f};

  for (int ks = ks_begin; ks < ks_end; ++ks) {
    const int wr = ks * 4 + kq;
    const bool ok = wr < kw;
    h8_t b[4];
    h8_t av[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int row = t * kTileM + j;
      u4_t xv = u4_t{0u, 0u, 0u, 0u};
      if (ok && row < a.M) xv = *(const u4_t*)(a.X + (int64_t)row * a.ldx + wr * 8);
      av[t] = __builtin_bit_cast(h8_t, xv);
    }
    if (ok && col_ok) {
      const int k0 = wr * 8;
      uint32_t g[8];
      if (ACT) {
        const u4_t g0 = *(const u4_t*)(a.g_idx + k0);
        const u4_t g1 = *(const u4_t*)(a.g_idx + k0 + 4);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          g[r] = min(g0[r], gmax);
          g[r + 4] = min(g1[r], gmax);
        }
      } else {
#pragma unroll
        for (int r = 0; r < 8; ++r) g[r] = (uint32_t)((k0 + r) / a.G);
      }
      const u4_t wv = *(const u4_t*)(a.qw + (int64_t)wr * a.ldq + col);
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const u2_t sv = *(const u2_t*)(a.sc + (int64_t)g[r] * a.lds + col);
        const uint32_t zw = a.qz[(int64_t)g[r] * a.ldz + (col >> 3)] >> zshift;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t q = (wv[c] >> (4 * r)) & 0xFu;
          const uint32_t z = (zw >> (4 * c)) & 0xFu;
          const _Float16 qz = __builtin_bit_cast(_Float16, (uint16_t)(0x6400u | q)) -
                              __builtin_bit_cast(_Float16, (uint16_t)(0x6400u | z));
          const _Float16 sc = __builtin_bit_cast(
              _Float16, (uint16_t)(((c < 2 ? sv.x : sv.y) >> (16 * (c & 1))) & 0xFFFFu));
          b[c][r] = qz * sc;
        }
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 8; ++r) b[c][r] = (_Float16)0.f;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[t][c] = mfma16x16x32(av[t], b[c], acc[t][c]);
  }
  finish_tile<MT>(a, acc, tile, split, red);
}

__global__ void k_gather_cols(const uint16_t* __restrict__ X, int64_t ldx, int M, int K,
                              const int32_t* __restrict__ perm, uint16_t* __restrict__ Xp) {
  const int64_t total = (int64_t)M * K;
  const uint32_t kmax = (uint32_t)(K - 1);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(i / K);
    const int jj = (int)(i - (int64_t)m * K);
    const uint32_t p = min((uint32_t)perm[jj], kmax);
    Xp[i] = X[(int64_t)m * ldx + p];
  }
}

int mtiles(int M) { return (M + kTileM - 1) / kTileM; }

}  // namespace

int decode_splits(int M, int K, int N) {
  const int ncol = (N + kDecodeCols - 1) / kDecodeCols;
  const int nks = (K + 31) / 32;
  // aim for ~2048 waves (8 per CU) but keep at least 2 k-steps per wave
  const int target_waves = 2048;
  int waves_per_tile = (target_waves + ncol - 1) / ncol;
  int splits = (waves_per_tile + kDecodeWaves - 1) / kDecodeWaves;
  const int max_splits = nks / (kDecodeWaves * 2);
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  (void)M;
  return splits;
}

size_t decode_ws_bytes(int M, int K, int N) {
  const int ncol = (N + kDecodeCols - 1) / kDecodeCols;
  const int splits = decode_splits(M, K, N);
  size_t b = align_up((size_t)ncol * 4);
  if (splits > 1) b += align_up((size_t)splits * M * N * 4);
  return b;
}

hipError_t launch_decode_ordered(const GemmArgs& a, hipStream_t s) {
  const int ncol = (a.N + kDecodeCols - 1) / kDecodeCols;
  dim3 grid(ncol * a.splits), block(256);
  switch (mtiles(a.M)) {
    case 1: hipLaunchKernelGGL(k_decode_ordered<1>, grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL(k_decode_ordered<2>, grid, block, 0, s, a); break;
    case 3:
    case 4: hipLaunchKernelGGL(k_decode_ordered<4>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_decode_rowmeta(const GemmArgs& a, bool actorder, hipStream_t s) {
  const int ncol = (a.N + kDecodeCols - 1) / kDecodeCols;
  dim3 grid(ncol * a.splits), block(256);
  const int mt = mtiles(a.M);
  if (actorder) {
    switch (mt) {
      case 1: hipLaunchKernelGGL((k_decode_rowmeta<1, true>), grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL((k_decode_rowmeta<2, true>), grid, block, 0, s, a); break;
      case 3:
      case 4: hipLaunchKernelGGL((k_decode_rowmeta<4, true>), grid, block, 0, s, a); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (mt) {
      case 1: hipLaunchKernelGGL((k_decode_rowmeta<1, false>), grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL((k_decode_rowmeta<2, false>), grid, block, 0, s, a); break;
      case 3:
      case 4: hipLaunchKernelGGL((k_decode_rowmeta<4, false>), grid, block, 0, s, a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_gather_cols(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                              uint16_t* Xp, hipStream_t s) {
  const int64_t total = (int64_t)M * K;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_gather_cols, dim3(blocks), dim3(256), 0, s, X, ldx, M, K, perm, Xp);
  return hipGetLastError();
}

}  // namespace tpdq
