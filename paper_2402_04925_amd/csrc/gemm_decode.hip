// W4A16 dequantize-and-multiply for decode-sized batches (M <= 64) on gfx950.
//
// Y[m][n] = sum_k X[m][k] * s[g(k)][n] * (q[k][n] - z[g(k)][n])
// (group quantization of section 1.1; g(k) = g_idx[k] under act-order, Eq. 3,
// or floor(k / G) for sorted rows, Eq. 1 after Alg. 1).
//
// Geometry. A workgroup owns 16 output columns over the whole K range, so no
// partial sums ever leave it (cross-workgroup reductions need agent-scope
// cache maintenance on the 8-XCD part, which costs more than the GEMM). Its
// NW waves split K into runs of 128-row blocks. Per 32-row step and lane
// (j = lane % 16, kq = lane / 16):
//   * B: the packed word of rows 32s + 8kq .. +7 of column j - the 8 fp16
//     B values of one lane of v_mfma_f32_16x16x32_f16 are exactly one word;
//   * A: 8 activations of row j of the row tile over the same 8 rows;
//   * one MFMA per 16-row tile of M.
// Latency: each wave issues the loads of its next blocks of weights before it
// computes the current ones; the tile's scales and zeros and the activations
// (X, or the gathered X[:, P1]) are staged in LDS while the first weight loads
// are in flight, so a workgroup waits for HBM about once.
// Issue rate: the kernel runs close to the VALU issue limit, so the
// activations are staged in LDS already in MFMA operand order (one 16-byte
// LDS read per step and tile, no shuffles) and the metadata pre-decoded.
//
// Metadata modes:
//   kMetaGroup (sorted rows, G % 32 == 0): a 32-row step lies inside one
//     group; the MFMAs accumulate sum_k x (q - z) exactly (q - z is a small
//     integer, exact in fp16) and the group's scale is applied once:
//     acc += s * group_acc. This is the metadata reuse of Fig. 2.
//   kMetaRowLds / kMetaRowGlobal (act-order): each of the 8 rows of a lane's
//     word takes its own group through g_idx (Fig. 1); the weight is
//     dequantized per element to fp16 before the MFMA. The tile's metadata is
//     staged in LDS, or fetched from global memory row by row.
#include "tpdq_internal.h"

namespace tpdq {
namespace {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ h2_t as_h2(uint32_t v) { return __builtin_bit_cast(h2_t, v); }
__device__ __forceinline__ uint32_t as_u32(h2_t v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ h8_t as_h8(u4_t v) { return __builtin_bit_cast(h8_t, v); }
// Takes the word by value: clang lowers __builtin_bit_cast applied directly to
// an ext_vector element (v.y) as a read of element 0.
__device__ __forceinline__ float as_f32(uint32_t v) { return __builtin_bit_cast(float, v); }

__device__ __forceinline__ float half_bits_to_float(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(bits16 & 0xFFFFu));
}

__device__ __forceinline__ uint16_t float_to_half_bits(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);  // round to nearest even
}

// Packed word -> 8 fp16 values (q - z) of one column, exact.
// OR-ing a nibble into the mantissa of 1024.0 (0x6400) gives 1024 + q; the
// nibbles at bits 4..7 land as 1024 + 16 q and are rescaled by 1/16 inside
// the same fused op. Order: k0, k4, k1, k5, k2, k6, k3, k7 (the A operand is
// staged in the same order).
// The masks live in VGPRs (v_and_or_b32 takes no two literals and reads one
// SGPR at most on this ISA), so each pair costs one v_and_or_b32.
struct UnpackConsts {
  uint32_t lo, hi, magic;
  __device__ __forceinline__ UnpackConsts() {
    asm volatile("v_mov_b32 %0, 0x000f000f" : "=v"(lo));
    asm volatile("v_mov_b32 %0, 0x00f000f0" : "=v"(hi));
    asm volatile("v_mov_b32 %0, 0x64006400" : "=v"(magic));
  }
};

__device__ __forceinline__ h8_t unpack_sub(const UnpackConsts& k, uint32_t w, uint32_t z1024,
                                           uint32_t z64) {
  const uint32_t lo = k.lo, hi = k.hi, magic = k.magic;
  const uint32_t w8 = w >> 8;
  const h2_t inv16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  u4_t r;
  r.x = as_u32(as_h2((w & lo) | magic) - as_h2(z1024));
  r.y = as_u32(as_h2((w & hi) | magic) * inv16 - as_h2(z64));
  r.z = as_u32(as_h2((w8 & lo) | magic) - as_h2(z1024));
  r.w = as_u32(as_h2((w8 & hi) | magic) * inv16 - as_h2(z64));
  return as_h8(r);
}


// Per-row dequant of one word: row r (0..7) has zero z[r] and scale bits
// s[r]; returns fp16(s * (q - z)) in the order k0, k4, k1, k5, k2, k6, k3, k7.
__device__ __forceinline__ h8_t dequant_rows(const UnpackConsts& k, uint32_t w,
                                             const uint32_t (&z)[8], const uint32_t (&s)[8]) {
  const uint32_t lo = k.lo, hi = k.hi, magic = k.magic;
  const uint32_t w8 = w >> 8;
  const h2_t inv16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  const uint32_t z04 = ((0x6400u | z[0]) | ((0x6400u | z[4]) << 16));
  const uint32_t z15 = ((0x5400u | (z[1] << 4)) | ((0x5400u | (z[5] << 4)) << 16));
  const uint32_t z26 = ((0x6400u | z[2]) | ((0x6400u | z[6]) << 16));
  const uint32_t z37 = ((0x5400u | (z[3] << 4)) | ((0x5400u | (z[7] << 4)) << 16));
  u4_t r;
  r.x = as_u32((as_h2((w & lo) | magic) - as_h2(z04)) * as_h2(s[0] | (s[4] << 16)));
  r.y = as_u32((as_h2((w & hi) | magic) * inv16 - as_h2(z15)) * as_h2(s[1] | (s[5] << 16)));
  r.z = as_u32((as_h2((w8 & lo) | magic) - as_h2(z26)) * as_h2(s[2] | (s[6] << 16)));
  r.w = as_u32((as_h2((w8 & hi) | magic) * inv16 - as_h2(z37)) * as_h2(s[3] | (s[7] << 16)));
  return as_h8(r);
}

// 8 consecutive fp16 activations x0..x7 -> x0, x4, x1, x5, x2, x6, x3, x7.
__device__ __forceinline__ u4_t permute_octet(u4_t x) {
  u4_t r;
  r.x = (x.x & 0xFFFFu) | (x.z << 16);
  r.y = (x.x >> 16) | (x.z & 0xFFFF0000u);
  r.z = (x.y & 0xFFFFu) | (x.w << 16);
  r.w = (x.y >> 16) | (x.w & 0xFFFF0000u);
  return r;
}

__device__ __forceinline__ f4_t mfma16x16x32(h8_t a, h8_t b, f4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Groups of the 8 rows of word row wr: g_idx when given, else floor(k / G)
// (sorted rows whose G is not a multiple of 32).
__device__ __forceinline__ void load_groups(const GemmArgs& a, bool ok, int wr, u4_t (&g)[2]) {
  if (!ok) {
    g[0] = u4_t{0u, 0u, 0u, 0u};
    g[1] = u4_t{0u, 0u, 0u, 0u};
  } else if (a.g_idx) {
    g[0] = *(const u4_t*)(a.g_idx + wr * 8);
    g[1] = *(const u4_t*)(a.g_idx + wr * 8 + 4);
  } else {
    const uint32_t k0 = (uint32_t)wr * 8u, G = (uint32_t)a.G;
    g[0] = u4_t{k0 / G, (k0 + 1) / G, (k0 + 2) / G, (k0 + 3) / G};
    g[1] = u4_t{(k0 + 4) / G, (k0 + 5) / G, (k0 + 6) / G, (k0 + 7) / G};
  }
}

// Workgroups are dispatched round-robin over the 8 XCDs. Neighbouring
// 16-column tiles share 128-byte lines of scales (and, in the GPTQ layout, of
// qweight), so consecutive tiles go to workgroups on the same XCD (same L2).
__device__ __forceinline__ int xcd_tile(int b, int nb) {
  if (nb % 8) return b;
  return (b % 8) * (nb / 8) + b / 8;
}

// ---------------------------------------------------------------------------
// Staging into LDS. Global loads go to registers before the weight stream is
// started, so waiting for them never waits for HBM; what does not fit in the
// registers is copied afterwards, four loads in flight at a time.
// ---------------------------------------------------------------------------

// Metadata of the 16-column tile, one 16-byte entry per (group, column):
//   DECODE 1 (kMetaGroup, subtracting zeros in the unpack):
//             {scale as fp32 bits, 1024 + z (fp16 x2), 64 + z (fp16 x2), 0}
//   DECODE 0 (kMetaRowLds): scale fp16 bits | z << 16 in the first word
template <int NT, int R, int DECODE>
struct MetaStage {
  uint32_t s[R], z[R];
  __device__ __forceinline__ void load(const GemmArgs& a, int n0, int rows, int tid) {
    const int items = rows * kTileN;
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int idx = tid + i * NT;
      const int n = n0 + (idx & 15);
      const int g = idx >> 4;
      const bool ok = idx < items && n < a.N;
      s[i] = ok ? (uint32_t)a.sc[(int64_t)g * a.lds + n] : 0u;
      z[i] = ok ? a.qz[(int64_t)g * a.ldz + (n >> 3)] : 0u;
    }
  }
  __device__ __forceinline__ static void put(u4_t* meta, int idx, int n, uint32_t sbits,
                                             uint32_t zw) {
    const uint32_t zc = (zw >> (4 * (n & 7))) & 0xFu;
    u4_t v;
    if (DECODE == 1) {
      v.x = __builtin_bit_cast(uint32_t, half_bits_to_float(sbits));
      v.y = (0x6400u | zc) * 0x10001u;
      v.z = (0x5400u | (zc << 4)) * 0x10001u;
      v.w = 0u;
    } else {
      v = u4_t{sbits | (zc << 16), 0u, 0u, 0u};
    }
    meta[idx] = v;
  }
  __device__ __forceinline__ void store(const GemmArgs& a, u4_t* meta, int n0, int rows, int tid) {
    const int items = rows * kTileN;
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int idx = tid + i * NT;
      if (idx < items) put(meta, idx, n0 + (idx & 15), s[i], z[i]);
    }
    for (int base = tid + R * NT; base < items; base += 4 * NT) {
      uint32_t ss[4], zz[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = base + i * NT;
        const int n = n0 + (idx & 15);
        const int g = idx >> 4;
        const bool ok = idx < items && n < a.N;
        ss[i] = ok ? (uint32_t)a.sc[(int64_t)g * a.lds + n] : 0u;
        zz[i] = ok ? a.qz[(int64_t)g * a.ldz + (n >> 3)] : 0u;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = base + i * NT;
        if (idx < items) put(meta, idx, n0 + (idx & 15), ss[i], zz[i]);
      }
    }
  }
};

// Activations in operand order: LDS entry (r * M + m) holds row m, rows
// 8r..8r+7 of the operand, permuted as x0, x4, x1, x5, x2, x6, x3, x7, for
// r < 16 * ceil(K / 128) (zero past K). With GATHER the operand column k is X
// column perm[k] (X[:, perm]). One more zero entry follows (see a_addr).
template <int NT, bool GATHER>
struct XStage {
  static constexpr int R = 4;
  u4_t v[R];   // !GATHER: raw 16-byte rows; GATHER: permutation entries
  __device__ __forceinline__ void load(const GemmArgs& a, int tid) {
    const int kw = a.K >> 3;
#pragma unroll
    for (int i = 0; i < R; ++i) {
      if (GATHER) {
        // entries of octet r = tid + (i/2)*NT, half i%2
        const int r = tid + (i >> 1) * NT;
        v[i] = r < kw ? *(const u4_t*)(a.perm + r * 8 + 4 * (i & 1)) : u4_t{0u, 0u, 0u, 0u};
      } else {
        const int m = i;  // rows 0..R-1 of octet tid (first pass)
        v[i] = (m < a.M && tid < kw) ? *(const u4_t*)(a.X + (int64_t)m * a.ldx + tid * 8)
                                     : u4_t{0u, 0u, 0u, 0u};
      }
    }
  }
  __device__ __forceinline__ static u4_t gather_octet(const GemmArgs& a, int m, const u4_t& p0,
                                                      const u4_t& p1) {
    const uint32_t kmax = (uint32_t)(a.K - 1);
    const uint16_t* xr = a.X + (int64_t)m * a.ldx;
    uint32_t x[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = xr[min(p0[e], kmax)];
      x[e + 4] = xr[min(p1[e], kmax)];
    }
    return u4_t{x[0] | (x[1] << 16), x[2] | (x[3] << 16), x[4] | (x[5] << 16), x[6] | (x[7] << 16)};
  }
  __device__ __forceinline__ void store(const GemmArgs& a, u4_t* xs, int tid) {
    const int kw = a.K >> 3;
    const int M = a.M;
    const int kwp = 16 * ((a.K + 127) >> 7);
    for (int i = kw * M + tid; i <= kwp * M; i += NT) xs[i] = u4_t{0u, 0u, 0u, 0u};
    if (GATHER) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = tid + h * NT;
        if (r < kw)
          for (int m = 0; m < M; ++m) xs[r * M + m] = permute_octet(gather_octet(a, m, v[2 * h], v[2 * h + 1]));
      }
      for (int r = tid + 2 * NT; r < kw; r += NT) {
        const u4_t p0 = *(const u4_t*)(a.perm + r * 8);
        const u4_t p1 = *(const u4_t*)(a.perm + r * 8 + 4);
        for (int m = 0; m < M; ++m) xs[r * M + m] = permute_octet(gather_octet(a, m, p0, p1));
      }
    } else {
      if (tid < kw) {
#pragma unroll
        for (int m = 0; m < R; ++m)
          if (m < M) xs[tid * M + m] = permute_octet(v[m]);
      }
      // the rest: rows >= R of the first pass, then further octets
      for (int m = 0; m < M; ++m) {
        for (int base = (m < R ? tid + NT : tid); base < kw; base += 4 * NT) {
          u4_t t4[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = base + i * NT;
            t4[i] = r < kw ? *(const u4_t*)(a.X + (int64_t)m * a.ldx + r * 8) : u4_t{0u, 0u, 0u, 0u};
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = base + i * NT;
            if (r < kw) xs[r * M + m] = permute_octet(t4[i]);
          }
        }
      }
    }
  }
};

// Sum the NW waves' 16-column partial tiles in LDS and write fp16.
// acc[t] of lane l holds rows t*16 + 4*(l/16) + e, column l % 16.
template <int MT, int NW>
__device__ __forceinline__ void reduce_store(const GemmArgs& a, f4_t (&acc)[MT], int n0,
                                             unsigned char* smem) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  __syncthreads();  // everyone is done with the staged operands
  float* red = (float*)smem;  // [NW][MT][4][64]
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[((wave * MT + t) * 4 + e) * 64 + lane] = acc[t][e];
  __syncthreads();
  for (int idx = tid; idx < MT * 256; idx += NW * 64) {
    const int t = idx >> 8;
    const int e = (idx >> 6) & 3;
    const int ln = idx & 63;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[((w * MT + t) * 4 + e) * 64 + ln];
    const int row = t * kTileM + 4 * (ln >> 4) + e;
    const int c = n0 + (ln & 15);
    if (row < a.M && c < a.N) a.Y[(int64_t)row * a.ldy + c] = float_to_half_bits(s);
  }
}

// Weights of one 128-row block (4 steps of 32 rows) for lane (j, kq) of
// column col: word u of the result = rows 32 (4b + u) + 8 kq .. +7.
template <int LAYOUT>
__device__ __forceinline__ u4_t load_block(const GemmArgs& a, const uint32_t* qcol,
                                           const uint32_t* qtile, int lane, int kq, int b,
                                           bool ok, int kw) {
  u4_t w = u4_t{0u, 0u, 0u, 0u};
  if (!ok) return w;
  if constexpr (LAYOUT == TPDQ_LAYOUT_TILED) {
    w = *(const u4_t*)(qtile + (int64_t)b * 256 + lane * 4);
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int wr = 4 * (4 * b + u) + kq;
      w[u] = wr < kw ? qcol[(int64_t)wr * a.ldq] : 0u;
    }
  }
  return w;
}

// A fragments of one block from global memory (rows t*16 + j, 8 halfs each),
// permuted into operand order unless the operand already is (kAGlobalPrep).
template <int MT, int AM>
__device__ __forceinline__ void load_a_block(const GemmArgs& a, int j, int kq, int b, bool ok,
                                             int kw, u4_t (&x)[4][MT]) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int wr = 4 * (4 * b + u) + kq;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int row = t * kTileM + j;
      const u4_t v = (ok && wr < kw && row < a.M)
                         ? *(const u4_t*)(a.X + (int64_t)row * a.ldx + wr * 8)
                         : u4_t{0u, 0u, 0u, 0u};
      x[u][t] = AM == kAGlobalPrep ? v : permute_octet(v);
    }
  }
}

constexpr bool a_global(int am) { return am == kAGlobal || am == kAGlobalPrep; }

// LDS entry of the A fragment of row tile t at step s for lane (j, kq):
// base + stride * s, with rows past M pointed at the zero entry (stride 0).
struct AAddr {
  int base, stride;
  __device__ __forceinline__ void init(int M, int j, int kq, int t, int zero_slot) {
    const int row = t * kTileM + j;
    const bool on = row < M;
    base = on ? kq * M + row : zero_slot;
    stride = on ? 4 * M : 0;
  }
};

// ---------------------------------------------------------------------------
// Ordered kernel: sorted rows, group of row k = k / G, G = 32 * SPG. Each wave
// owns a run of 128-row blocks; CB blocks of weights are prefetched one chunk
// ahead. Group boundaries inside a block sit at compile-time positions.
// ---------------------------------------------------------------------------
template <int MT, int NW, int SPG, int AM, int LAYOUT>
__global__ __launch_bounds__(NW * 64) void k_ordered(GemmArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NT = NW * 64;
  constexpr bool AG = a_global(AM);
  constexpr int CB = AG ? (MT == 1 ? 2 : 1) : 4;  // blocks per chunk
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int n0 = tile * kTileN;
  const int col = n0 + j;
  const bool col_ok = col < a.N;
  const int kw = a.K >> 3;
  const int ng = a.K / (32 * SPG);
  const int nsteps = a.K >> 5;  // 32-row steps
  const int nblk = (a.K + 127) >> 7;
  const int b0 = (int)((int64_t)nblk * wave / NW);
  const int b1 = (int)((int64_t)nblk * (wave + 1) / NW);
  u4_t* meta = (u4_t*)smem;
  u4_t* xs = (u4_t*)(smem + a.lds_x_off);
  const int zero_slot = a.M * 16 * nblk;  // the zero entry after the staged X
  const uint32_t* qcol = a.qw + col;
  const uint32_t* qtile = a.qw + (int64_t)tile * a.ldq;
  const bool wok = LAYOUT == TPDQ_LAYOUT_TILED ? true : col_ok;
  const UnpackConsts kc;

  // 1. staging loads (L2-resident) into registers
  MetaStage<NT, 4, 1> ms;
  ms.load(a, n0, ng, tid);
  XStage<NT, AM == kALdsGather> xst;
  if constexpr (!AG) xst.load(a, tid);

  // 2. the weight stream: first chunk
  u4_t wb[CB];
  u4_t ab[AG ? CB : 1][4][MT];
#pragma unroll
  for (int bi = 0; bi < CB; ++bi) {
    const bool ok = b0 + bi < b1;
    wb[bi] = load_block<LAYOUT>(a, qcol, qtile, lane, kq, b0 + bi, ok && wok, kw);
    if constexpr (AG) load_a_block<MT, AM>(a, j, kq, b0 + bi, ok, kw, ab[bi]);
  }

  // 3. staged operands to LDS
  ms.store(a, meta, n0, ng, tid);
  if constexpr (!AG) xst.store(a, xs, tid);
  __syncthreads();

  // 4. main loop
  AAddr aa[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) aa[t].init(a.M, j, kq, t, zero_slot);
  f4_t acc[MT], gacc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    acc[t] = f4_t{0.f, 0.f, 0.f, 0.f};
    gacc[t] = f4_t{0.f, 0.f, 0.f, 0.f};
  }
  const f4_t fz = {0.f, 0.f, 0.f, 0.f};
  float s_cur = 0.f;
  uint32_t z1024 = 0x64006400u, z64 = 0x54005400u;
  auto set_group = [&](int g) {
    const u4_t v = meta[min(g, ng - 1) * kTileN + j];
    s_cur = as_f32(v.x);
    z1024 = v.y;
    z64 = v.z;
  };
  // close a group: acc += s * group_acc
  auto flush = [&]() {
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] += s_cur * gacc[t];
  };
  set_group((4 * b0) / SPG);
  bool open = false;  // a group has been accumulated and not yet closed
  for (int c = b0; c < b1; c += CB) {
    u4_t wn[CB];
    u4_t an[AG ? CB : 1][4][MT];
    const bool more = c + CB < b1;
    if (more) {
#pragma unroll
      for (int bi = 0; bi < CB; ++bi) {
        const bool ok = c + CB + bi < b1;
        wn[bi] = load_block<LAYOUT>(a, qcol, qtile, lane, kq, c + CB + bi, ok && wok, kw);
        if constexpr (AG) load_a_block<MT, AM>(a, j, kq, c + CB + bi, ok, kw, an[bi]);
      }
    }
#pragma unroll
    for (int bi = 0; bi < CB; ++bi) {
      const int b = c + bi;
      if (b < b1) {
        h8_t av[4][MT];
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          const int i0 = aa[t].base + aa[t].stride * (4 * b);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if constexpr (AG)
              av[u][t] = as_h8(ab[bi][u][t]);
            else
              av[u][t] = as_h8(xs[i0 + aa[t].stride * u]);
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          // K is a multiple of G and so of 32: the steps of a partial last
          // block past K hold no rows and must not reopen the last group
          if (4 * b + u >= nsteps) break;
          bool start;
          if constexpr (SPG <= 4)
            start = (u % SPG) == 0;
          else
            start = u == 0 && (b % (SPG / 4)) == 0;
          if (start) {  // a new group begins at this step: close the last one
            if (open) flush();
            set_group((4 * b + u) / SPG);
          }
          open = true;
          const h8_t bv = unpack_sub(kc, wb[bi][u], z1024, z64);
#pragma unroll
          for (int t = 0; t < MT; ++t) gacc[t] = mfma16x16x32(av[u][t], bv, start ? fz : gacc[t]);
        }
      }
    }
    if (more) {
#pragma unroll
      for (int bi = 0; bi < CB; ++bi) {
        wb[bi] = wn[bi];
        if constexpr (AG) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int t = 0; t < MT; ++t) ab[bi][u][t] = an[bi][u][t];
        }
      }
    }
  }
  if (open) flush();
  reduce_store<MT, NW>(a, acc, n0, smem);
}

// ---------------------------------------------------------------------------
// Row-metadata kernel: each of the 8 rows of a word looks its group up
// (g_idx, or floor(k / G) when g_idx is NULL) and is dequantized on its own.
// One 128-row block of weights (and of g_idx) is prefetched ahead.
// ---------------------------------------------------------------------------
template <int MT, int NW, int META, int AM, int LAYOUT>
__global__ __launch_bounds__(NW * 64) void k_rowmeta(GemmArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NT = NW * 64;
  constexpr bool AG = a_global(AM);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int n0 = tile * kTileN;
  const int col = n0 + j;
  const bool col_ok = col < a.N;
  const int kw = a.K >> 3;
  const int nblk = (a.K + 127) >> 7;
  const int b0 = (int)((int64_t)nblk * wave / NW);
  const int b1 = (int)((int64_t)nblk * (wave + 1) / NW);
  u4_t* meta = (u4_t*)smem;
  u4_t* xs = (u4_t*)(smem + a.lds_x_off);
  const int zero_slot = a.M * 16 * nblk;
  const uint32_t* qcol = a.qw + col;
  const uint32_t* qtile = a.qw + (int64_t)tile * a.ldq;
  const bool wok = LAYOUT == TPDQ_LAYOUT_TILED ? true : col_ok;
  const UnpackConsts kc;

  MetaStage<NT, 8, 0> ms;
  if constexpr (META == kMetaRowLds) ms.load(a, n0, a.meta_rows, tid);
  XStage<NT, false> xst;
  if constexpr (!AG) xst.load(a, tid);

  auto load_g = [&](int b, u4_t (&g)[4][2]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int wr = 4 * (4 * b + u) + kq;
      load_groups(a, b < b1 && wr < kw, wr, g[u]);
    }
  };
  u4_t wb = load_block<LAYOUT>(a, qcol, qtile, lane, kq, b0, b0 < b1 && wok, kw);
  u4_t gb[4][2];
  load_g(b0, gb);
  u4_t ab[4][MT];
  if constexpr (AG) load_a_block<MT, AM>(a, j, kq, b0, b0 < b1, kw, ab);

  if constexpr (META == kMetaRowLds) ms.store(a, meta, n0, a.meta_rows, tid);
  if constexpr (!AG) xst.store(a, xs, tid);
  if constexpr (META == kMetaRowLds || !AG) __syncthreads();
  AAddr aa[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) aa[t].init(a.M, j, kq, t, zero_slot);

  f4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f4_t{0.f, 0.f, 0.f, 0.f};
  const uint32_t gmax = (uint32_t)(a.num_groups - 1);
  const int zshift = 4 * (col & 7);
  for (int b = b0; b < b1; ++b) {
    const bool more = b + 1 < b1;
    u4_t wn = u4_t{0u, 0u, 0u, 0u};
    u4_t gn[4][2];
    u4_t an[4][MT];
    if (more) {
      wn = load_block<LAYOUT>(a, qcol, qtile, lane, kq, b + 1, wok, kw);
      load_g(b + 1, gn);
      if constexpr (AG) load_a_block<MT, AM>(a, j, kq, b + 1, true, kw, an);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int wr = 4 * (4 * b + u) + kq;
      h8_t av[MT];
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        if constexpr (AG)
          av[t] = as_h8(ab[u][t]);
        else
          av[t] = as_h8(xs[aa[t].base + aa[t].stride * (4 * b + u)]);
      }
      uint32_t zr[8], sr[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const uint32_t g = min(r < 4 ? gb[u][0][r] : gb[u][1][r - 4], gmax);
        if constexpr (META == kMetaRowLds) {
          const uint32_t v = meta[g * kTileN + j].x;
          zr[r] = v >> 16;
          sr[r] = v & 0xFFFFu;
        } else {
          sr[r] = col_ok ? (uint32_t)a.sc[(int64_t)g * a.lds + col] : 0u;
          zr[r] = col_ok ? (a.qz[(int64_t)g * a.ldz + (col >> 3)] >> zshift) & 0xFu : 0u;
        }
      }
      const h8_t bv = dequant_rows(kc, wb[u], zr, sr);
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[t] = mfma16x16x32(av[t], bv, acc[t]);
    }
    if (more) {
      wb = wn;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        gb[u][0] = gn[u][0];
        gb[u][1] = gn[u][1];
      }
      if constexpr (AG) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int t = 0; t < MT; ++t) ab[u][t] = an[u][t];
      }
    }
  }
  reduce_store<MT, NW>(a, acc, n0, smem);
}

// X'[m][k] = X[m][perm[k]] (perm NULL: X itself), written in operand order
// (each 8-column octet permuted as x0, x4, x1, x5, x2, x6, x3, x7) for
// kAGlobalPrep.
__global__ void k_gather_prep(const uint16_t* __restrict__ X, int64_t ldx, int M, int K,
                              const int32_t* __restrict__ perm, uint16_t* __restrict__ Xp) {
  const int kw = K >> 3;
  const int64_t total = (int64_t)M * kw;
  const uint32_t kmax = (uint32_t)(K - 1);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(i / kw);
    const int r = (int)(i - (int64_t)m * kw);
    const uint16_t* xr = X + (int64_t)m * ldx;
    uint32_t x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      x[e] = xr[perm ? min((uint32_t)perm[r * 8 + e], kmax) : (uint32_t)(r * 8 + e)];
    const u4_t v = {x[0] | (x[4] << 16), x[1] | (x[5] << 16), x[2] | (x[6] << 16),
                    x[3] | (x[7] << 16)};
    *(u4_t*)(Xp + (int64_t)m * K + r * 8) = v;
  }
}

typedef void (*DecodeKernel)(GemmArgs);

template <int MT, int NW, int SPG, int L>
DecodeKernel pick_ordered_am(int am) {
  switch (am) {
    case kAGlobal: return k_ordered<MT, NW, SPG, kAGlobal, L>;
    case kAGlobalPrep: return k_ordered<MT, NW, SPG, kAGlobalPrep, L>;
    case kALds: return k_ordered<MT, NW, SPG, kALds, L>;
    case kALdsGather: return k_ordered<MT, NW, SPG, kALdsGather, L>;
  }
  return nullptr;
}

template <int MT, int NW, int L>
DecodeKernel pick_ordered_spg(int spg, int am) {
  switch (spg) {
    case 1: return pick_ordered_am<MT, NW, 1, L>(am);
    case 2: return pick_ordered_am<MT, NW, 2, L>(am);
    case 4: return pick_ordered_am<MT, NW, 4, L>(am);
    case 8: return pick_ordered_am<MT, NW, 8, L>(am);
  }
  return nullptr;
}

template <int MT, int NW, int L, int META>
DecodeKernel pick_row_am(int am) {
  switch (am) {
    case kAGlobal: return k_rowmeta<MT, NW, META, kAGlobal, L>;
    case kAGlobalPrep: return k_rowmeta<MT, NW, META, kAGlobalPrep, L>;
    case kALds: return k_rowmeta<MT, NW, META, kALds, L>;
  }
  return nullptr;
}

template <int MT, int NW, int L>
DecodeKernel pick_mt_nw(const DecodePlan& p) {
  if (p.meta == kMetaGroup) return pick_ordered_spg<MT, NW, L>(p.spg, p.amode);
  if constexpr (NW <= 8) {
    if (p.meta == kMetaRowLds) return pick_row_am<MT, NW, L, kMetaRowLds>(p.amode);
    return pick_row_am<MT, NW, L, kMetaRowGlobal>(p.amode);
  }
  return nullptr;
}

template <int MT, int L>
DecodeKernel pick_nw(const DecodePlan& p) {
  switch (p.nw) {
    case 4: return pick_mt_nw<MT, 4, L>(p);
    case 8: return pick_mt_nw<MT, 8, L>(p);
    case 16:
      if constexpr (MT < 4) return pick_mt_nw<MT, 16, L>(p);
      return nullptr;
  }
  return nullptr;
}

template <int L>
DecodeKernel pick_layout(const DecodePlan& p) {
  switch (p.mt) {
    case 1: return pick_nw<1, L>(p);
    case 2: return pick_nw<2, L>(p);
    case 4: return pick_nw<4, L>(p);
  }
  return nullptr;
}

DecodeKernel pick_kernel(const DecodePlan& p) {
  if (p.layout == TPDQ_LAYOUT_TILED) return pick_layout<TPDQ_LAYOUT_TILED>(p);
  return pick_layout<TPDQ_LAYOUT_GPTQ>(p);
}

}  // namespace

bool plan_decode(int M, int K, int N, int G, int num_groups, int layout, int meta_pref, int operand,
                 DecodePlan* p) {
  if (M < 1 || M > kDecodeMaxM) return false;
  const int mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  const int ntiles = (N + kTileN - 1) / kTileN;
  // waves per workgroup: about 16 resident waves per CU over the grid
  int nw = 16;
  if (ntiles > 256) nw = 8;
  if (ntiles > 1024) nw = 4;
  int meta = meta_pref;
  const int spg = G / 32;
  if (meta == kMetaGroup &&
      (G % 32 != 0 || K % G != 0 || !(spg == 1 || spg == 2 || spg == 4 || spg == 8)))
    meta = kMetaRowLds;  // sorted rows of another G: per-row groups floor(k / G)
  if ((meta != kMetaGroup || mt == 4) && nw > 8) nw = 8;
  int meta_rows = 0;
  if (meta == kMetaGroup) meta_rows = K / G;
  if (meta == kMetaRowLds) meta_rows = num_groups;
  const size_t red = (size_t)nw * mt * 1024;
  size_t meta_bytes = align_up((size_t)meta_rows * kTileN * 16, 16);
  if (meta_bytes > kLdsMax - red) {
    if (meta == kMetaGroup) return false;
    meta = kMetaRowGlobal;
    meta_rows = 0;
    meta_bytes = 0;
  }
  const size_t x_bytes = ((size_t)M * 16 * ((K + 127) / 128) + 1) * 16;  // padded + zero entry
  // stage X in LDS when it leaves room for two workgroups per CU (or one,
  // when the grid has no more workgroups than CUs)
  const size_t budget = ntiles <= 256 ? kLdsMax : kLdsMax / 2;
  const bool fits = meta_bytes + x_bytes <= budget;
  int am;
  if (operand == kOperandGather) {
    if (!fits || meta != kMetaGroup) return false;
    am = kALdsGather;
  } else if (operand == kOperandPrepared) {
    am = kAGlobalPrep;
  } else {
    am = fits ? kALds : kAGlobal;
  }
  p->layout = layout;
  p->meta = meta;
  p->amode = am;
  p->nw = nw;
  p->mt = mt;
  p->spg = spg;
  p->meta_rows = meta_rows;
  p->lds_x_off = (int)meta_bytes;
  size_t need = a_global(am) ? meta_bytes : meta_bytes + x_bytes;  // <= budget when staged
  if (need < red) need = red;
  p->lds_bytes = need;
  return pick_kernel(*p) != nullptr;
}

hipError_t launch_decode(const GemmArgs& a0, const DecodePlan& p, hipStream_t s) {
  DecodeKernel k = pick_kernel(p);
  if (!k) return hipErrorInvalidValue;
  GemmArgs a = a0;
  a.meta_rows = p.meta_rows;
  a.lds_x_off = p.lds_x_off;
  if (p.lds_bytes > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)kLdsMax);
    if (e != hipSuccess) return e;
  }
  const int ntiles = (a.N + kTileN - 1) / kTileN;
  hipLaunchKernelGGL(k, dim3(ntiles), dim3(p.nw * 64), p.lds_bytes, s, a);
  return hipGetLastError();
}

hipError_t launch_gather_prep(const uint16_t* X, int64_t ldx, int M, int K, const int32_t* perm,
                              uint16_t* Xp, hipStream_t s) {
  const int64_t total = (int64_t)M * (K / 8);
  int blocks = (int)((total + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_gather_prep, dim3(blocks), dim3(256), 0, s, X, ldx, M, K, perm, Xp);
  return hipGetLastError();
}

}  // namespace tpdq
