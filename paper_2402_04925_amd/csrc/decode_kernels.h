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
//
// Element type DT (fp16 or bf16 activations, scales and outputs). With bf16
// the ordered kernels take B = 128 + q exactly (unpack_bias_bf16) and close
// each group with s * (group_acc - (128 + z) * sum_k x), sum_k x from one more
// MFMA against ones per step and row tile; the per-row kernel dequantizes to
// bf16 through fp32.
#pragma once

#include "kernels_common.h"

namespace tpdq {
namespace {

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

// ---------------------------------------------------------------------------
// Staging into LDS. Global loads go to registers before the weight stream is
// started, so waiting for them never waits for HBM; what does not fit in the
// registers is copied afterwards, four loads in flight at a time.
// ---------------------------------------------------------------------------

// Metadata of the 16-column tile (kMetaRowLds), one 16-byte entry per
// (group, column): the scale's bits | z << 16 in word COMP (0; the gated
// kernel's up projection in word 1).
template <int NT, int R, int COMP = 0>
struct MetaStage {
  uint32_t s[R], z[R];
  // Entry idx = 16 g + c: group g, column n0 + c. The loads are branch-free:
  // group and column are clamped into the tile's metadata (entries past the
  // last group are never stored; columns past N meet zero weights or are not
  // written), so the weight loads issued behind them keep their own counts.
  __device__ __forceinline__ static void fetch(const GemmArgs& a, int n0, int rows, int idx,
                                               uint32_t& sv, uint32_t& zv) {
    const int g = min(idx >> 4, rows - 1);
    const int n = min(n0 + (idx & 15), a.N - 1);
    sv = a.sc[(int64_t)g * a.lds + n];
    zv = a.qz[(int64_t)g * a.ldz + (n >> 3)];
  }
  __device__ __forceinline__ void load(const GemmArgs& a, int n0, int rows, int tid) {
#pragma unroll
    for (int i = 0; i < R; ++i) fetch(a, n0, rows, tid + i * NT, s[i], z[i]);
  }
  // the stored zero code plus the layer's offset (up to 16) in the high half
  __device__ __forceinline__ static void put(u4_t* meta, int idx, int n, uint32_t sbits,
                                             uint32_t zw, int zoff) {
    const uint32_t zc = ((zw >> (4 * (n & 7))) & 0xFu) + (uint32_t)zoff;
    ((uint32_t*)&meta[idx])[COMP] = sbits | (zc << 16);
  }
  // Entries past the last group go to the spare entry meta[items], so every
  // value loaded in load() is consumed on every path (a value used only
  // under a branch lets the compiler sink its load behind the weight loads).
  __device__ __forceinline__ void store(const GemmArgs& a, u4_t* meta, int n0, int rows, int tid) {
    const int items = rows * kTileN;
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int idx = tid + i * NT;
      put(meta, min(idx, items), n0 + (idx & 15), s[i], z[i], a.zoff);
    }
    for (int base = tid + R * NT; base < items; base += 4 * NT) {
      uint32_t ss[4], zz[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) fetch(a, n0, rows, base + i * NT, ss[i], zz[i]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = base + i * NT;
        if (idx < items) put(meta, idx, n0 + (idx & 15), ss[i], zz[i], a.zoff);
      }
      wait_vmcnt<0>();  // no load of this loop outlives it (see wait_vmcnt)
    }
  }
};

// Activations in operand order: LDS entry (r * M + m) holds row m, rows
// 8r..8r+7 of the operand (permuted as x0, x4, x1, x5, x2, x6, x3, x7 for
// GPTQ weights, as they are for tiled ones), for r < 16 * ceil(K / 128)
// (zero past K). One more zero entry follows (see
// AAddr), then a spare entry. With GATHER the operand column k is X column
// perm[k] (X[:, perm]): the rows of X are first copied to LDS (at xr) and
// gathered from there, so no global load waits on another. With 2 <= M <= 4
// (and every piece of X held in registers) the copy is column-major, four
// halves per column (rows 0..3, zero past M), so one 8-byte LDS read
// fetches a column of every row; otherwise it is row-major, [M][K].
// Global loads are buffer loads: octets past K load zeros at no cost and go
// to a spare entry.
template <int NT, bool GATHER, int LAYOUT>
struct XStage {
  static constexpr int R = 8;
  // Slot s holds the 16 bytes of row m, octet r = tid + i * NT, stepping
  // (m, i) through rows 0..M-1 and passes 0..P-1, P = ceil(kw / NT): the
  // bookkeeping is wave-uniform, no per-lane division.
  __amdgpu_buffer_rsrc_t rx;
  u4_t v[R];
  u4_t p[2];   // GATHER: permutation entries of octet tid
  __device__ __forceinline__ u4_t piece(const GemmArgs& a, int m, int r, int kw) const {
    const uint32_t off = r < kw ? ((uint32_t)m * (uint32_t)a.ldx + (uint32_t)r * 8u) * 2u
                                : kOutOfRange;
    return buffer_load16(rx, off);
  }
  __device__ __forceinline__ void load(const GemmArgs& a, int tid) {
    const int kw = a.K >> 3;
    const int P = (kw + NT - 1) / NT;
    rx = buffer_rsrc(a.X, (uint32_t)a.M * (uint32_t)a.ldx * 2u);
    int m = 0, i = 0;
#pragma unroll
    for (int sl = 0; sl < R; ++sl) {
      if (m < a.M) v[sl] = piece(a, m, tid + i * NT, kw);
      if (++i == P) {
        i = 0;
        ++m;
      }
    }
    if (GATHER) {
      const __amdgpu_buffer_rsrc_t rp = buffer_rsrc(a.perm, (uint32_t)a.K * 4u);
      const uint32_t off = tid < kw ? (uint32_t)tid * 32u : kOutOfRange;
      p[0] = buffer_load16(rp, off);
      p[1] = buffer_load16(rp, off + 16u);
    }
  }
  // row m, octet r to its operand entry, or (GATHER) to the LDS copy of X;
  // octets past K go to the spare entry (xs[spare] or xr[M * kw])
  __device__ __forceinline__ static void put(u4_t* xs, u4_t* xr, int M, int kw, int spare, int m,
                                             int r, const u4_t& x) {
    if (GATHER)
      xr[r < kw ? m * kw + r : M * kw] = x;
    else
      xs[r < kw ? r * M + m : spare] = to_operand<LAYOUT>(x);
  }
  // column-major copy of X: octet r = tid + I NT of rows 0..3 (pieces in
  // slots m P + I, zeros past M) as eight 8-byte columns at xr + 4 r
  template <int SL>
  __device__ __forceinline__ u4_t slot(bool on) const {
    if constexpr (SL < R) return on ? v[SL] : u4_t{0u, 0u, 0u, 0u};
    return u4_t{0u, 0u, 0u, 0u};
  }
  template <int P, int I>
  __device__ __forceinline__ void store_colmajor(u4_t* xr, int M, int kw, int tid) const {
    if constexpr (I < P) {
      const u4_t row[4] = {slot<I>(true), slot<P + I>(M > 1), slot<2 * P + I>(M > 2),
                           slot<3 * P + I>(M > 3)};
      const int r = tid + I * NT;
      u4_t* dst = xr + 4 * (r < kw ? r : kw);  // octets past K: the spare columns
#pragma unroll
      for (int w = 0; w < 4; ++w)  // columns 2w, 2w + 1
        dst[w] = u4_t{__builtin_amdgcn_perm(row[1][w], row[0][w], 0x05040100u),
                      __builtin_amdgcn_perm(row[3][w], row[2][w], 0x05040100u),
                      __builtin_amdgcn_perm(row[1][w], row[0][w], 0x07060302u),
                      __builtin_amdgcn_perm(row[3][w], row[2][w], 0x07060302u)};
      store_colmajor<P, I + 1>(xr, M, kw, tid);
    }
  }
  static __device__ __forceinline__ bool colmajor(int M, int kw) {
    const int P = (kw + NT - 1) / NT;
    return GATHER && M >= 2 && M <= 4 && M * P <= R;
  }
  __device__ __forceinline__ void store(const GemmArgs& a, u4_t* xs, u4_t* xr, int tid) {
    const int kw = a.K >> 3;
    const int M = a.M;
    const int P = (kw + NT - 1) / NT;
    const int kwp = 16 * ((a.K + 127) >> 7);
    const int spare = kwp * M + 1;  // after the zero entry
    for (int e = kw * M + tid; e <= kwp * M; e += NT) xs[e] = u4_t{0u, 0u, 0u, 0u};
    if (GATHER && colmajor(M, kw)) {
      switch (P) {
        case 1: store_colmajor<1, 0>(xr, M, kw, tid); break;
        case 2: store_colmajor<2, 0>(xr, M, kw, tid); break;
        case 3: store_colmajor<3, 0>(xr, M, kw, tid); break;
        default: store_colmajor<4, 0>(xr, M, kw, tid); break;
      }
      __syncthreads();  // the copy of X is complete
      const uint32_t kmax = (uint32_t)(a.K - 1);
      const unsigned char* xb = (const unsigned char*)xr;
      for (int r = tid; r < kw; r += NT) {
        u4_t p0 = p[0], p1 = p[1];
        if (r != tid) {
          p0 = *(const u4_t*)(a.perm + r * 8);
          p1 = *(const u4_t*)(a.perm + r * 8 + 4);
          wait_vmcnt<0>();
        }
        uint32_t q[8][2];  // column perm[8 r + e]: rows 0, 1 in q[e][0], rows 2, 3 in q[e][1]
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t c = min(e < 4 ? p0[e] : p1[e - 4], kmax);
          const uint2 t = *(const uint2*)(xb + 8u * c);
          q[e][0] = t.x;
          q[e][1] = t.y;
        }
#pragma unroll
        for (int mr = 0; mr < 4; ++mr) {
          if (mr >= M) break;
          const uint32_t sel = (mr & 1) ? 0x07060302u : 0x05040100u;
          const int h = mr >> 1;
          xs[r * M + mr] = to_operand<LAYOUT>(u4_t{__builtin_amdgcn_perm(q[1][h], q[0][h], sel),
                                                   __builtin_amdgcn_perm(q[3][h], q[2][h], sel),
                                                   __builtin_amdgcn_perm(q[5][h], q[4][h], sel),
                                                   __builtin_amdgcn_perm(q[7][h], q[6][h], sel)});
        }
      }
      return;
    }
    int m = 0, i = 0;
#pragma unroll
    for (int sl = 0; sl < R; ++sl) {
      if (m < M) put(xs, xr, M, kw, spare, m, tid + i * NT, v[sl]);
      if (++i == P) {
        i = 0;
        ++m;
      }
    }
    // what did not fit in the registers, four loads in flight at a time
    while (m < M) {
      u4_t t4[4];
      int mm[4], rr[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        mm[q] = m;
        rr[q] = tid + i * NT;
        t4[q] = m < M ? piece(a, m, rr[q], kw) : u4_t{0u, 0u, 0u, 0u};
        if (++i == P) {
          i = 0;
          ++m;
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (mm[q] < M) put(xs, xr, M, kw, spare, mm[q], rr[q], t4[q]);
      wait_vmcnt<0>();  // no load of this loop outlives it (see wait_vmcnt)
    }
    if (GATHER) {
      __syncthreads();  // the copy of X is complete
      const uint16_t* x16 = (const uint16_t*)xr;
      const uint32_t kmax = (uint32_t)(a.K - 1);
      for (int r = tid; r < kw; r += NT) {
        u4_t p0 = p[0], p1 = p[1];
        if (r != tid) {
          p0 = *(const u4_t*)(a.perm + r * 8);
          p1 = *(const u4_t*)(a.perm + r * 8 + 4);
          wait_vmcnt<0>();
        }
        uint32_t c[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          c[e] = min(p0[e], kmax);
          c[e + 4] = min(p1[e], kmax);
        }
        for (int mr = 0; mr < M; ++mr) {
          const uint16_t* xm = x16 + mr * a.K;
          xs[r * M + mr] = to_operand<LAYOUT>(u4_t{xm[c[0]] | ((uint32_t)xm[c[1]] << 16),
                                                   xm[c[2]] | ((uint32_t)xm[c[3]] << 16),
                                                   xm[c[4]] | ((uint32_t)xm[c[5]] << 16),
                                                   xm[c[6]] | ((uint32_t)xm[c[7]] << 16)});
        }
      }
    }
  }
};

// Offset (in elements) of Y[row][c] in the prepared-operand layout of a
// following GEMM whose K is this GEMM's N (the records of k_gather_prep:
// [row tile][step][lane] x 8 values, rows 8 (4 step + lane / 16) .. +7 of
// the operand for row 16 tile + lane % 16, in natural order for tiled
// weights, else x0, x4, x1, x5, ...).
__device__ __forceinline__ int64_t prepared_offset(int row, int c, int nsteps, int natural) {
  const int r = c >> 3, e = c & 7;
  const int64_t rec = ((int64_t)(row >> 4) * nsteps + (r >> 2)) * 64 + 16 * (r & 3) + (row & 15);
  return rec * 8 + (natural ? e : (e & 3) * 2 + (e >> 2));
}

// Sum the NW waves' partial tiles (TN tiles of 16 columns from n0) in LDS
// and write Y in the element type; with a.Yp, Y is also written in the next
// GEMM's prepared-operand layout (a.N a multiple of 128: no padding).
// acc[t][n] of lane l holds rows t*16 + 4*(l/16) + e, column n0 + 16 n +
// l % 16. GATED: tiles 0 and 1 are the gate and up products of the same 16
// columns, and Y = silu(gate) * up (in fp32, rounded once).
template <int MT, int NW, int TN, int DT, bool GATED = false>
__device__ __forceinline__ void reduce_store(const GemmArgs& a, f4_t (&acc)[MT][TN], int n0,
                                             unsigned char* smem) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  __syncthreads();  // everyone is done with the staged operands
  float* red = (float*)smem;  // [NW][MT][TN][4][64]
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int n = 0; n < TN; ++n)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        red[(((wave * MT + t) * TN + n) * 4 + e) * 64 + lane] = acc[t][n][e];
  __syncthreads();
  if constexpr (GATED) {
    // tile 0 holds X W_gate, tile 1 X W_up, both for columns n0 .. n0 + 15
    for (int idx = tid; idx < MT * 256; idx += NW * 64) {
      const int t = idx >> 8;
      const int e = (idx >> 6) & 3;
      const int ln = idx & 63;
      float g = 0.f, u = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        g += red[((w * MT * TN + t * TN + 0) * 4 + e) * 64 + ln];
        u += red[((w * MT * TN + t * TN + 1) * 4 + e) * 64 + ln];
      }
      const int row = t * kTileM + 4 * (ln >> 4) + e;
      const int c = n0 + (ln & 15);
      if (row < a.M && c < a.N) {
        const uint16_t v = float_to_bits<DT>(g / (1.f + __expf(-g)) * u);  // silu(g) * u
        a.Y[(int64_t)row * a.ldy + c] = v;
        if (a.Yp) a.Yp[prepared_offset(row, c, a.N >> 5, a.yp_natural)] = v;
      }
    }
    return;
  }
  for (int idx = tid; idx < MT * TN * 256; idx += NW * 64) {
    const int tn = idx >> 8;  // t * TN + n
    const int e = (idx >> 6) & 3;
    const int ln = idx & 63;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[((w * MT * TN + tn) * 4 + e) * 64 + ln];
    const int row = (tn / TN) * kTileM + 4 * (ln >> 4) + e;
    const int c = n0 + (tn % TN) * kTileN + (ln & 15);
    if (row < a.M && c < a.N) {
      const uint16_t v = float_to_bits<DT>(s);
      a.Y[(int64_t)row * a.ldy + c] = v;
      if (a.Yp) a.Yp[prepared_offset(row, c, a.N >> 5, a.yp_natural)] = v;
    }
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
// in operand order (the prepared operand already is).
template <int MT, int AM, int LAYOUT>
__device__ __forceinline__ void load_a_block(const GemmArgs& a, int j, int kq, int b, bool ok,
                                             int kw, u4_t (&x)[4][MT]) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int wr = 4 * (4 * b + u) + kq;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int row = t * kTileM + j;
      if constexpr (AM == kAGlobalPrep) {
        // the prepared operand's record [t][4b + u][16 kq + j] (see k_gather_prep)
        const int64_t nsteps = 4 * (int64_t)((a.K + 127) >> 7);
        const int64_t rec = ((int64_t)t * nsteps + 4 * b + u) * 64 + 16 * kq + j;
        x[u][t] = ok ? *(const u4_t*)(a.X + rec * 8) : u4_t{0u, 0u, 0u, 0u};
      } else {
        const u4_t v = (ok && wr < kw && row < a.M)
                           ? *(const u4_t*)(a.X + (int64_t)row * a.ldx + wr * 8)
                           : u4_t{0u, 0u, 0u, 0u};
        x[u][t] = to_operand<LAYOUT>(v);
      }
    }
  }
}

constexpr bool a_global(int am) { return am == kAGlobal || am == kAGlobalPrep; }

// The weight stream of one 16-column tile: block b (128 rows) for lane
// (j, kq); word u = rows 32 (4b + u) + 8 kq .. +7 of column n0 + j.
// Tiled: one 16-byte load per block. GPTQ: four 4-byte loads (rows past K
// read zeros; columns past N read whatever lies there and are not written).
template <int LAYOUT>
struct WeightStream {
  __amdgpu_buffer_rsrc_t rs;
  uint32_t lane_off;   // byte offset of the lane's data in block 0
  uint32_t blk_bytes;  // bytes between consecutive blocks
  // tile_ok false (a tile past N): every load returns zeros
  __device__ __forceinline__ void init(const GemmArgs& a, int tile, bool tile_ok, int lane, int kq,
                                       int col, int nblk) {
    if constexpr (LAYOUT == TPDQ_LAYOUT_TILED) {
      rs = buffer_rsrc(a.qw + (int64_t)tile * a.ldq, tile_ok ? (uint32_t)nblk * 1024u : 0u);
      lane_off = (uint32_t)lane * 16u;
      blk_bytes = 1024u;
    } else {
      rs = buffer_rsrc(a.qw, tile_ok ? (uint32_t)(a.K >> 3) * (uint32_t)a.ldq * 4u : 0u);
      lane_off = ((uint32_t)kq * (uint32_t)a.ldq + (uint32_t)col) * 4u;
      blk_bytes = 16u * (uint32_t)a.ldq * 4u;
    }
  }
  // block b if valid, else zeros at no cost
  __device__ __forceinline__ u4_t fetch(int b, bool valid, int64_t ldq) const {
    const uint32_t base = valid ? (uint32_t)b * blk_bytes + lane_off : kOutOfRange;
    if constexpr (LAYOUT == TPDQ_LAYOUT_TILED) {
      return buffer_load16<kNonTemporal>(rs, base);
    } else {
      const uint32_t step = 4u * (uint32_t)ldq * 4u;  // 32 rows = 4 word rows
      u4_t w;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        w[u] = buffer_load4<kNonTemporal>(rs, valid ? base + u * step : kOutOfRange);
      return w;
    }
  }
};

// A fragments of block b from global memory: row t*16 + j, rows 8 (4 (4b + u)
// + kq) .. +7, as stored (for GPTQ weights the consumer permutes them into
// operand order unless they already are, kAGlobalPrep: permuting at the load
// would make the load be waited for at once).
// Rows past M read zeros from the resource bound; columns past K are zeroed.
// kAGlobalPrep reads the prepared operand (k_gather_prep): 16-byte records
// [row tile t][step s][lane], one contiguous KiB per load instruction, in
// operand order and zero-padded.
template <int MT, int AM>
struct AStream {
  __amdgpu_buffer_rsrc_t rs;
  uint32_t row_off[MT];
  __device__ __forceinline__ AStream(const GemmArgs& a, int j, int lane) {
    if constexpr (AM == kAGlobalPrep) {
      const uint32_t nsteps = 4u * (uint32_t)((a.K + 127) >> 7);
      rs = buffer_rsrc(a.X, (uint32_t)MT * nsteps * 1024u);
      // rows past M hold zeros: skip them (out of range loads cost nothing)
#pragma unroll
      for (int t = 0; t < MT; ++t)
        row_off[t] = t * kTileM + j < a.M ? ((uint32_t)t * nsteps * 64u + (uint32_t)lane) * 16u
                                          : kOutOfRange;
    } else {
      rs = buffer_rsrc(a.X, (uint32_t)a.M * (uint32_t)a.ldx * 2u);
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int row = t * kTileM + j;
        row_off[t] = row < a.M ? (uint32_t)row * (uint32_t)a.ldx * 2u : kOutOfRange;
      }
    }
  }
  __device__ __forceinline__ void fetch(int b, bool valid, int kq, int kw, u4_t (&x)[4][MT]) const {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int wr = 4 * (4 * b + u) + kq;
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        uint32_t off;
        if constexpr (AM == kAGlobalPrep)
          off = valid && row_off[t] != kOutOfRange ? row_off[t] + (uint32_t)(4 * b + u) * 1024u
                                                   : kOutOfRange;
        else
          off = valid && wr < kw && row_off[t] != kOutOfRange ? row_off[t] + (uint32_t)wr * 16u
                                                              : kOutOfRange;
        x[u][t] = buffer_load16(rs, off);  // raw: permuted where it is used
      }
    }
  }
};



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

// Scales and zeros of the ordered kernel, per wave and per chunk of 4 blocks
// (16 steps of 32 rows, groups g0 = 16 c / (4 SPG) onwards). They travel with
// the weight stream instead of through LDS, so no wave waits for another
// wave's metadata: lane 16 q + j loads group g0 + 4 n + q (set n < NL) of
// column n0 + j, decodes it once per chunk, and a lane that opens group g
// reads it from lane 16 ((g - g0) % 4) + j of set (g - g0) / 4 (ds_bpermute).
template <int SPG, int DT>
struct ChunkMeta {
  static constexpr int NL = SPG >= 4 ? 1 : 4 / SPG;
  __amdgpu_buffer_rsrc_t rs, rz;
  uint32_t soff, zoff;    // this lane's pair in group row g0 = 0
  uint32_t sgrp, zgrp;    // bytes per group row
  uint32_t shift;         // nibble of column n0 + j in its zeros word
  uint32_t zadd;          // the layer's zero offset, added to each zero code
  uint32_t raw_s[NL], raw_z[NL];
  float s[NL];
  uint32_t z1024[NL], z64[NL];
  __device__ __forceinline__ void init(const GemmArgs& a, int ng, int col, int q) {
    rs = buffer_rsrc(a.sc, (uint32_t)ng * (uint32_t)a.lds * 2u);
    rz = buffer_rsrc(a.qz, (uint32_t)ng * (uint32_t)a.ldz * 4u);
    sgrp = (uint32_t)a.lds * 2u;
    zgrp = (uint32_t)a.ldz * 4u;
    soff = (uint32_t)q * sgrp + (uint32_t)col * 2u;
    zoff = (uint32_t)q * zgrp + (uint32_t)(col >> 3) * 4u;
    shift = 4u * (uint32_t)(col & 7);
    zadd = (uint32_t)a.zoff;
  }
  // the chunk whose first group is g0 (groups past ng load zeros)
  __device__ __forceinline__ void load(int g0, bool valid, int ng, int q) {
#pragma unroll
    for (int n = 0; n < NL; ++n) {
      const bool ok = valid && g0 + 4 * n + q < ng;
      const uint32_t g = (uint32_t)(g0 + 4 * n);
      raw_s[n] = buffer_load2(rs, ok ? soff + g * sgrp : kOutOfRange);
      raw_z[n] = buffer_load4(rz, ok ? zoff + g * zgrp : kOutOfRange);
    }
  }
  // {scale as fp32, 1024 + z (fp16 x2), 64 + z (fp16 x2)}, see unpack_sub;
  // bf16: {scale as fp32, 128 + z as fp32 bits, unused}
  __device__ __forceinline__ void decode() {
#pragma unroll
    for (int n = 0; n < NL; ++n) {
      const uint32_t zc = ((raw_z[n] >> shift) & 0xFu) + zadd;  // up to 16
      s[n] = bits_to_float<DT>(raw_s[n]);
      if constexpr (DT == kBF16) {
        z1024[n] = __builtin_bit_cast(uint32_t, 128.f + (float)zc);
        z64[n] = 0u;
      } else {
        z1024[n] = (0x6400u | zc) * 0x10001u;
        z64[n] = (0x5400u | (zc << 4)) * 0x10001u;
      }
    }
  }
  __device__ __forceinline__ void get(int n, int src, float& sv, uint32_t& z1, uint32_t& z2) const {
    sv = __shfl(s[n], src);
    z1 = (uint32_t)__shfl((int)z1024[n], src);
    z2 = (uint32_t)__shfl((int)z64[n], src);
  }
};

// ---------------------------------------------------------------------------
// Ordered kernel: sorted rows, group of row k = k / G, G = 32 * SPG. A
// workgroup owns TN 16-column tiles over all of K (TN = 2 halves the
// activation traffic per column where X is read from global memory). Each
// wave owns a run of 128-row blocks and keeps D of them in flight: the loads
// are issued in the order the blocks are consumed and waited for one block at
// a time, so the dequant and MFMAs of a block run while later blocks are
// still arriving. Each chunk's scales and zeros are loaded just before its
// first block. Block ranges and the loop are wave-uniform (scalar); group
// boundaries inside a chunk sit at compile-time positions for G <= 128.
// ---------------------------------------------------------------------------
template <int MT, int NW, int SPG, int AM, int LAYOUT, int TN, int DT, bool GATED = false>
__global__ __launch_bounds__(NW * 64) void k_ordered(GemmArgs a) {
  // GATED: one 16-column tile, its TN = 2 weight streams are the gate and up
  // projections (same shape and leading dimensions), Y = silu(gate) * up
  static_assert(!GATED || TN == 2, "the gated kernel streams gate and up");
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NT = NW * 64;
  constexpr bool AG = a_global(AM);
  // 128-row blocks in flight per wave; with A from global memory its
  // fragments (4 * MT registers of 16 bytes per block) ride along. The
  // prepared operand with one row tile keeps four (Llama-70B TP=8 MLP at
  // M = 8: 16.1 -> 14.6 us; at M = 16 equal, 17.1 us), the other global
  // operands two, or one with four row tiles
  constexpr int D = AG ? (MT == 4 ? 1 : (AM == kAGlobalPrep && MT == 1 && !GATED ? 4 : 2)) : 4;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int tile0 = xcd_tile(blockIdx.x, gridDim.x) * (GATED ? 1 : TN);
  const int ntiles = (a.N + kTileN - 1) / kTileN;
  const int kw = a.K >> 3;
  const int ng = (a.K + 32 * SPG - 1) / (32 * SPG);  // the last group may be partial
  const int nblk = (a.K + 127) >> 7;
  const int b0 = (int)((int64_t)nblk * wave / NW);
  const int b1 = (int)((int64_t)nblk * (wave + 1) / NW);
  GemmArgs au = a;  // stream n's weights: the up projection's for n = 1 when GATED
  if constexpr (GATED) {
    au.qw = a.qw_up;
    au.sc = a.sc_up;
    au.qz = a.qz_up;
  }
  auto tile_of = [&](int n) { return GATED ? tile0 : tile0 + n; };
  u4_t* xs = (u4_t*)(smem + a.lds_x_off);
  u4_t* xr = (u4_t*)(smem + a.lds_xr_off);
  const int zero_slot = a.M * 16 * nblk;  // the zero entry after the staged X
  const UnpackConsts<DT> kc;

  // 1. loads, in the order they are needed: activations (L2 hits, staged in
  //    LDS), the first chunk's scales and zeros, the first D weight blocks
  //    (the scheduling barriers keep that issue order: loads complete in
  //    order, so a load moved behind the weights would be waited for last)
  XStage<NT, AM == kALdsGather, LAYOUT> xst;
  if constexpr (!AG) xst.load(a, tid);
  __builtin_amdgcn_sched_barrier(0);
  ChunkMeta<SPG, DT> cm[TN];
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    cm[n].init(GATED && n == 1 ? au : a, ng, tile_of(n) * kTileN + j, kq);
    cm[n].load((4 * b0) / SPG, b0 < b1, ng, kq);
  }
  __builtin_amdgcn_sched_barrier(0);
  WeightStream<LAYOUT> wsrc[TN];
#pragma unroll
  for (int n = 0; n < TN; ++n)
    wsrc[n].init(GATED && n == 1 ? au : a, tile_of(n), tile_of(n) < ntiles, lane, kq,
                 tile_of(n) * kTileN + j, nblk);
  const AStream<MT, AM> asrc(a, j, lane);
  u4_t wb[D][TN];
  u4_t ab[AG ? D : 1][4][MT];
  auto fetch = [&](int b, int slot) {
#pragma unroll
    for (int n = 0; n < TN; ++n) wb[slot][n] = wsrc[n].fetch(b, b < b1, a.ldq);
    if constexpr (AG) asrc.fetch(b, b < b1, kq, kw, ab[slot]);
  };
#pragma unroll
  for (int i = 0; i < D; ++i) {
    fetch(b0 + i, i);
    __builtin_amdgcn_sched_barrier(0);
  }

  // 2. activations to LDS; the metadata and weights stay in flight
  if constexpr (!AG) {
    xst.store(a, xs, xr, tid);
    wait_vmcnt<TN * (2 * ChunkMeta<SPG, DT>::NL + D * (LAYOUT == TPDQ_LAYOUT_TILED ? 1 : 4))>();
    __syncthreads();
  }

  // 3. main loop
  AAddr aa[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) aa[t].init(a.M, j, kq, t, zero_slot);
  f4_t acc[MT][TN], gacc[MT][TN];
  f4_t xsum[MT];  // bf16: sum of the group's activations per row
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    xsum[t] = f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int n = 0; n < TN; ++n) {
      acc[t][n] = f4_t{0.f, 0.f, 0.f, 0.f};
      gacc[t][n] = f4_t{0.f, 0.f, 0.f, 0.f};
    }
  }
  const f4_t fz = {0.f, 0.f, 0.f, 0.f};
  const u4_t ones = {kBf16OnePair, kBf16OnePair, kBf16OnePair, kBf16OnePair};
  float s_cur[TN];
  uint32_t z1024[TN], z64[TN];
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    s_cur[n] = 0.f;
    z1024[n] = 0x64006400u;
    z64[n] = 0x54005400u;
  }

  // block c + i of the chunk starting at block c: 4 steps of 32 rows; a group
  // opens at its first step (fresh MFMA accumulator, its scale and zeros) and
  // closes at its last (acc += s * group_acc). Steps past K have zero
  // activations and groups past the last one zero metadata.
  auto block = [&](int c, int i, const u4_t (&w)[TN], const u4_t (&av_g)[4][MT]) {
    const int b = c + i;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int st = 4 * b + u;
      bool open, close;
      if constexpr (SPG <= 4) {
        open = (u % SPG) == 0;
        close = (u % SPG) == SPG - 1;
      } else {  // SPG == 8: a group is blocks 2g and 2g + 1
        open = u == 0 && ((b & 1) == 0 || b == b0);
        close = u == 3 && ((b & 1) == 1 || b == b1 - 1);
      }
      if (open) {
#pragma unroll
        for (int n = 0; n < TN; ++n) {
          if constexpr (SPG <= 4) {
            const int rel = (4 * i + u) / SPG;  // compile-time once unrolled
            cm[n].get(rel >> 2, 16 * (rel & 3) + j, s_cur[n], z1024[n], z64[n]);
          } else {
            const int rel = st / SPG - (4 * c) / SPG;  // 0..2
            cm[n].get(0, 16 * rel + j, s_cur[n], z1024[n], z64[n]);
          }
        }
      }
      u4_t av[MT];
#pragma unroll
      for (int t = 0; t < MT; ++t)
        av[t] = AG ? (AM == kAGlobalPrep ? av_g[u][t] : to_operand<LAYOUT>(av_g[u][t]))
                   : xs[aa[t].base + aa[t].stride * st];
#pragma unroll
      for (int n = 0; n < TN; ++n) {
        const u4_t bv = unpack_step<DT>(kc, w[n][u], z1024[n], z64[n]);
#pragma unroll
        for (int t = 0; t < MT; ++t)
          gacc[t][n] = mfma_k32<DT>(av[t], bv, open ? fz : gacc[t][n]);
      }
      if constexpr (DT == kBF16) {
#pragma unroll
        for (int t = 0; t < MT; ++t) xsum[t] = mfma_k32<DT>(av[t], ones, open ? fz : xsum[t]);
      }
      if (close) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
          for (int n = 0; n < TN; ++n) {
            if constexpr (DT == kBF16)
              acc[t][n] += s_cur[n] * (gacc[t][n] - as_f32(z1024[n]) * xsum[t]);
            else
              acc[t][n] += s_cur[n] * gacc[t][n];
          }
      }
    }
  };

  // Every load is unconditional (a block or group past the run loads zeros
  // for free), so that each use waits for exactly what it needs: a load
  // behind a branch makes the wait counts fall back to waiting for all.
  for (int c = b0; c < b1; c += 4) {
#pragma unroll
    for (int n = 0; n < TN; ++n) {
      cm[n].decode();
      cm[n].load((4 * (c + 4)) / SPG, c + 4 < b1, ng, kq);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int b = c + i;
      if (b < b1) block(c, i, wb[i % D], ab[AG ? i % D : 0]);
      fetch(b + D, i % D);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  reduce_store<MT, NW, TN, DT, GATED>(a, acc, tile0 * kTileN, smem);
}


// ---------------------------------------------------------------------------
// Wide kernel (large weights, X too large to stage whole in LDS): the
// workgroup's NW waves own NW * TN different 16-column tiles
// over one range of 128-row blocks of K (all of K, or one of ks splits), so
// that the activations are shared: they are staged in LDS four blocks at a
// time (two buffers, loaded with the LDS bit, one barrier per chunk) while
// each wave streams its own weights in registers, D blocks ahead, and owns
// its outputs (no cross-wave reduction). With ks > 1 each workgroup writes
// its fp32 partial tile to a.part[split][M][N] (k_splitk_reduce adds them).
// PREP: the activations are the prepared operand (k_gather_prep records),
// else X row-major.
// ---------------------------------------------------------------------------
template <int MT, int NW, int SPG, int TN, bool PREP, int DT>
__global__ __launch_bounds__(NW * 64) void k_wide(GemmArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int D = 4;                  // weight blocks in flight per wave
  constexpr int CB = 4;                 // blocks per activation chunk
  constexpr int RECS = MT * CB * 4;     // 1 KiB operand records per chunk
  static_assert(RECS % NW == 0, "records split evenly over the waves");
  constexpr int RPW = RECS / NW;
  constexpr int CHUNK = RECS * 1024;    // bytes per LDS buffer
  constexpr int NL = ChunkMeta<SPG, DT>::NL;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15;
  const int kq = lane >> 4;
  const int ks = a.ks > 1 ? a.ks : 1;
  const int wgs = (int)(gridDim.x / ks);  // workgroups per split
  const int lt = xcd_tile(blockIdx.x, gridDim.x);
  const int kidx = lt / wgs;
  const int tg = lt - kidx * wgs;
  const int tile0 = (tg * NW + wave) * TN;  // this wave's first tile
  const int ntiles = (a.N + kTileN - 1) / kTileN;
  const int ng = (a.K + 32 * SPG - 1) / (32 * SPG);  // the last group may be partial
  const int nblk = (a.K + 127) >> 7;
  const int kw = a.K >> 3;
  const int b0 = (int)((int64_t)nblk * kidx / ks);
  const int b1 = (int)((int64_t)nblk * (kidx + 1) / ks);
  const UnpackConsts<DT> kc;

  // activation records: record r of a chunk is (row tile t, step sl) =
  // (r / (4 CB), r % (4 CB)), stored at r KiB of the buffer; lane l holds
  // row 16 t + l % 16, rows 8 (4 st + l / 16) .. +7 of the operand
  __amdgpu_buffer_rsrc_t rx;
  uint32_t x_lane, x_t, x_st;
  if constexpr (PREP) {
    const uint32_t nst = 4u * (uint32_t)nblk;
    rx = buffer_rsrc(a.X, (uint32_t)((a.M + 15) / 16) * nst * 1024u);
    x_lane = (uint32_t)lane * 16u;
    x_t = nst * 1024u;
    x_st = 1024u;
  } else {
    rx = buffer_rsrc(a.X, (uint32_t)a.M * (uint32_t)a.ldx * 2u);
    x_lane = ((uint32_t)j * (uint32_t)a.ldx + 8u * (uint32_t)kq) * 2u;
    x_t = 16u * (uint32_t)a.ldx * 2u;
    x_st = 64u;
  }
  auto issue_a = [&](int cb0, int buf) {
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
      const int r = wave * RPW + i;
      const int t = r / (4 * CB), sl = r % (4 * CB);
      const int st = 4 * cb0 + sl;
      // the lane's octet 4 st + kq: octets past K load zeros (a partial last
      // step when K % 32 != 0; the padding of X past K is never read)
      uint32_t off = 4 * st + kq < kw ? x_lane + (uint32_t)t * x_t + (uint32_t)st * x_st : kOutOfRange;
      asm("" : "+v"(off));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rx, (__attribute__((address_space(3))) void*)(smem + buf * CHUNK + r * 1024), 16, off, 0,
          0, 0);
    }
  };

  ChunkMeta<SPG, DT> cm[TN];
  WeightStream<TPDQ_LAYOUT_TILED> wsrc[TN];
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    cm[n].init(a, ng, (tile0 + n) * kTileN + j, kq);
    wsrc[n].init(a, tile0 + n, tile0 + n < ntiles, lane, kq, (tile0 + n) * kTileN + j, nblk);
  }
  u4_t wb[D][TN];
  auto fetch = [&](int b, int slot) {
#pragma unroll
    for (int n = 0; n < TN; ++n) wb[slot][n] = wsrc[n].fetch(b, b < b1, a.ldq);
  };

  // prologue, in the order the loads are needed
  issue_a(b0, 0);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int n = 0; n < TN; ++n) cm[n].load((4 * b0) / SPG, b0 < b1, ng, kq);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < D; ++i) {
    fetch(b0 + i, i);
    __builtin_amdgcn_sched_barrier(0);
  }

  f4_t acc[MT][TN], gacc[MT][TN];
  f4_t xsum[MT];  // bf16: sum of the group's activations per row
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    xsum[t] = f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int n = 0; n < TN; ++n) {
      acc[t][n] = f4_t{0.f, 0.f, 0.f, 0.f};
      gacc[t][n] = f4_t{0.f, 0.f, 0.f, 0.f};
    }
  }
  const f4_t fz = {0.f, 0.f, 0.f, 0.f};
  const u4_t ones = {kBf16OnePair, kBf16OnePair, kBf16OnePair, kBf16OnePair};
  float s_cur[TN];
  uint32_t z1024[TN], z64[TN];
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    s_cur[n] = 0.f;
    z1024[n] = 0x64006400u;
    z64[n] = 0x54005400u;
  }

  // block c + i, its activations in LDS buffer `buf`
  auto block = [&](int c, int i, int buf, const u4_t (&w)[TN]) {
    const int b = c + i;
    const u4_t* ab = (const u4_t*)(smem + buf * CHUNK);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int st = 4 * b + u;
      bool open, close;
      if constexpr (SPG <= 4) {
        open = (u % SPG) == 0;
        close = (u % SPG) == SPG - 1;
      } else {  // SPG == 8: a group is blocks 2g and 2g + 1
        open = u == 0 && ((b & 1) == 0 || b == b0);
        close = u == 3 && ((b & 1) == 1 || b == b1 - 1);
      }
      if (open) {
#pragma unroll
        for (int n = 0; n < TN; ++n) {
          if constexpr (SPG <= 4) {
            const int rel = (4 * i + u) / SPG;
            cm[n].get(rel >> 2, 16 * (rel & 3) + j, s_cur[n], z1024[n], z64[n]);
          } else {
            const int rel = st / SPG - (4 * c) / SPG;
            cm[n].get(0, 16 * rel + j, s_cur[n], z1024[n], z64[n]);
          }
        }
      }
      u4_t av[MT];
#pragma unroll
      for (int t = 0; t < MT; ++t) av[t] = ab[(t * 4 * CB + 4 * i + u) * 64 + lane];
#pragma unroll
      for (int n = 0; n < TN; ++n) {
        const u4_t bv = unpack_step<DT>(kc, w[n][u], z1024[n], z64[n]);
#pragma unroll
        for (int t = 0; t < MT; ++t)
          gacc[t][n] = mfma_k32<DT>(av[t], bv, open ? fz : gacc[t][n]);
      }
      if constexpr (DT == kBF16) {
#pragma unroll
        for (int t = 0; t < MT; ++t) xsum[t] = mfma_k32<DT>(av[t], ones, open ? fz : xsum[t]);
      }
      if (close) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
          for (int n = 0; n < TN; ++n) {
            if constexpr (DT == kBF16)
              acc[t][n] += s_cur[n] * (gacc[t][n] - as_f32(z1024[n]) * xsum[t]);
            else
              acc[t][n] += s_cur[n] * gacc[t][n];
          }
      }
    }
  };

  // Chunk c (blocks c .. c + 3): its activations were loaded with the LDS
  // bit before the metadata of this chunk and the D = 4 weight fetches that
  // followed, and loads complete in order; after the barrier every wave's
  // records of chunk c are in LDS and every wave is done with chunk c - 4's
  // buffer, which receives chunk c + 4.
  int buf = 0;
  for (int c = b0; c < b1; c += CB) {
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"(TN * (2 * NL + D))
                 : "memory");
    issue_a(c + CB, buf ^ 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int n = 0; n < TN; ++n) {
      cm[n].decode();
      cm[n].load((4 * (c + 4)) / SPG, c + 4 < b1, ng, kq);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int b = c + i;
      if (b < b1) block(c, i, buf, wb[i % D]);
      fetch(b + D, i % D);
      __builtin_amdgcn_sched_barrier(0);
    }
    buf ^= 1;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // each wave owns its columns: acc[t][n] of lane (j, kq) holds rows
  // 16 t + 4 kq .. +3, column 16 (tile0 + n) + j
  float* part = a.part + (size_t)kidx * a.M * a.N;
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int n = 0; n < TN; ++n) {
      const int col = (tile0 + n) * kTileN + j;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = t * kTileM + 4 * kq + e;
        if (row < a.M && col < a.N) {
          if (ks > 1)
            part[(int64_t)row * a.N + col] = acc[t][n][e];
          else
            a.Y[(int64_t)row * a.ldy + col] = float_to_bits<DT>(acc[t][n][e]);
        }
      }
    }
}

// ---------------------------------------------------------------------------
// Row-metadata kernel: each of the 8 rows of a word looks its group up
// (g_idx, or floor(k / G) when g_idx is NULL) and is dequantized on its own.
// One 128-row block of weights (and of g_idx) is prefetched ahead.
// ---------------------------------------------------------------------------
template <int MT, int NW, int META, int AM, int LAYOUT, int DT, bool GATED = false>
__global__ __launch_bounds__(NW * 64) void k_rowmeta(GemmArgs a) {
  // GATED: a second weight stream and metadata (the up projection, same
  // shape, leading dimensions and g_idx), Y = silu(X W) * (X W_up)
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
  const UnpackConsts<DT> kc;
  GemmArgs au = a;
  if constexpr (GATED) {
    au.qw = a.qw_up;
    au.sc = a.sc_up;
    au.qz = a.qz_up;
  }
  const uint32_t* qcol_u = au.qw + col;
  const uint32_t* qtile_u = au.qw + (int64_t)tile * a.ldq;

  MetaStage<NT, 8> ms;
  MetaStage<NT, 8, 1> msu;
  if constexpr (META == kMetaRowLds) ms.load(a, n0, a.meta_rows, tid);
  if constexpr (META == kMetaRowLds && GATED) msu.load(au, n0, a.meta_rows, tid);
  XStage<NT, false, LAYOUT> xst;
  if constexpr (!AG) xst.load(a, tid);

  auto load_g = [&](int b, u4_t (&g)[4][2]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int wr = 4 * (4 * b + u) + kq;
      load_groups(a, b < b1 && wr < kw, wr, g[u]);
    }
  };
  u4_t wb = load_block<LAYOUT>(a, qcol, qtile, lane, kq, b0, b0 < b1 && wok, kw);
  u4_t wbu = u4_t{0u, 0u, 0u, 0u};
  if constexpr (GATED) wbu = load_block<LAYOUT>(a, qcol_u, qtile_u, lane, kq, b0, b0 < b1 && wok, kw);
  u4_t gb[4][2];
  load_g(b0, gb);
  u4_t ab[4][MT];
  if constexpr (AG) load_a_block<MT, AM, LAYOUT>(a, j, kq, b0, b0 < b1, kw, ab);

  if constexpr (META == kMetaRowLds) ms.store(a, meta, n0, a.meta_rows, tid);
  if constexpr (META == kMetaRowLds && GATED) msu.store(au, meta, n0, a.meta_rows, tid);
  if constexpr (!AG) xst.store(a, xs, nullptr, tid);
  if constexpr (META == kMetaRowLds || !AG) __syncthreads();
  AAddr aa[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) aa[t].init(a.M, j, kq, t, zero_slot);

  f4_t acc[MT], accu[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    acc[t] = f4_t{0.f, 0.f, 0.f, 0.f};
    accu[t] = f4_t{0.f, 0.f, 0.f, 0.f};
  }
  const uint32_t gmax = (uint32_t)(a.num_groups - 1);
  const int zshift = 4 * (col & 7);
  const uint32_t zoff = (uint32_t)a.zoff;
  for (int b = b0; b < b1; ++b) {
    const bool more = b + 1 < b1;
    u4_t wn = u4_t{0u, 0u, 0u, 0u};
    u4_t wnu = u4_t{0u, 0u, 0u, 0u};
    u4_t gn[4][2];
    u4_t an[4][MT];
    if (more) {
      wn = load_block<LAYOUT>(a, qcol, qtile, lane, kq, b + 1, wok, kw);
      if constexpr (GATED) wnu = load_block<LAYOUT>(a, qcol_u, qtile_u, lane, kq, b + 1, wok, kw);
      load_g(b + 1, gn);
      if constexpr (AG) load_a_block<MT, AM, LAYOUT>(a, j, kq, b + 1, true, kw, an);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      u4_t av[MT];
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        if constexpr (AG)
          av[t] = ab[u][t];
        else
          av[t] = xs[aa[t].base + aa[t].stride * (4 * b + u)];
      }
      uint32_t zr[8], sr[8], zru[8], sru[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const uint32_t g = min(r < 4 ? gb[u][0][r] : gb[u][1][r - 4], gmax);
        if constexpr (META == kMetaRowLds) {
          if constexpr (GATED) {
            const uint2 v = *(const uint2*)&meta[g * kTileN + j];
            zr[r] = v.x >> 16;
            sr[r] = v.x & 0xFFFFu;
            zru[r] = v.y >> 16;
            sru[r] = v.y & 0xFFFFu;
          } else {
            const uint32_t v = meta[g * kTileN + j].x;
            zr[r] = v >> 16;
            sr[r] = v & 0xFFFFu;
          }
        } else {
          sr[r] = col_ok ? (uint32_t)a.sc[(int64_t)g * a.lds + col] : 0u;
          zr[r] = col_ok ? ((a.qz[(int64_t)g * a.ldz + (col >> 3)] >> zshift) & 0xFu) + zoff : 0u;
          if constexpr (GATED) {
            sru[r] = col_ok ? (uint32_t)au.sc[(int64_t)g * a.lds + col] : 0u;
            zru[r] = col_ok ? ((au.qz[(int64_t)g * a.ldz + (col >> 3)] >> zshift) & 0xFu) + zoff : 0u;
          }
        }
      }
      const u4_t bv = dequant_rows<LAYOUT == TPDQ_LAYOUT_TILED, DT>(kc, wb[u], zr, sr);
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[t] = mfma_k32<DT>(av[t], bv, acc[t]);
      if constexpr (GATED) {
        const u4_t bvu = dequant_rows<LAYOUT == TPDQ_LAYOUT_TILED, DT>(kc, wbu[u], zru, sru);
#pragma unroll
        for (int t = 0; t < MT; ++t) accu[t] = mfma_k32<DT>(av[t], bvu, accu[t]);
      }
    }
    if (more) {
      wb = wn;
      if constexpr (GATED) wbu = wnu;
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
  if constexpr (GATED) {
    f4_t acc2[MT][2];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      acc2[t][0] = acc[t];
      acc2[t][1] = accu[t];
    }
    reduce_store<MT, NW, 2, DT, true>(a, acc2, n0, smem);
  } else {
    f4_t acc1[MT][1];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc1[t][0] = acc[t];
    reduce_store<MT, NW, 1, DT>(a, acc1, n0, smem);
  }
}

// Kernel selection for a plan (DecodeKernel is declared with DecodePlan).
// Each dtype is instantiated in its own translation unit.
template <int MT, int NW, int SPG, int L, int DT>
DecodeKernel pick_ordered_am(int am, int tn) {
  // plan_decode gives the ordered kernel 4 or 8 waves and one tile with X in
  // LDS, 4 waves and one or two tiles with X from global memory; only those
  // are instantiated
  switch (am) {
    case kAGlobal:
      if constexpr (NW == 4)
        return tn == 2 ? k_ordered<MT, NW, SPG, kAGlobal, L, 2, DT> : k_ordered<MT, NW, SPG, kAGlobal, L, 1, DT>;
      return nullptr;
    case kAGlobalPrep:
      if constexpr (NW == 4)
        return tn == 2 ? k_ordered<MT, NW, SPG, kAGlobalPrep, L, 2, DT>
                       : k_ordered<MT, NW, SPG, kAGlobalPrep, L, 1, DT>;
      return nullptr;
    case kALds:
      if constexpr (NW <= 8) return tn == 1 ? k_ordered<MT, NW, SPG, kALds, L, 1, DT> : nullptr;
      return nullptr;
    case kALdsGather:
      if constexpr (NW <= 8) return tn == 1 ? k_ordered<MT, NW, SPG, kALdsGather, L, 1, DT> : nullptr;
      return nullptr;
  }
  return nullptr;
}

template <int MT, int NW, int L, int DT>
DecodeKernel pick_ordered_spg(int spg, int am, int tn) {
  switch (spg) {
    case 1: return pick_ordered_am<MT, NW, 1, L, DT>(am, tn);
    case 2: return pick_ordered_am<MT, NW, 2, L, DT>(am, tn);
    case 4: return pick_ordered_am<MT, NW, 4, L, DT>(am, tn);
    case 8: return pick_ordered_am<MT, NW, 8, L, DT>(am, tn);
  }
  return nullptr;
}

template <int MT, int NW, int L, int META, int DT>
DecodeKernel pick_row_am(int am) {
  switch (am) {
    case kAGlobal: return k_rowmeta<MT, NW, META, kAGlobal, L, DT>;
    case kAGlobalPrep: return k_rowmeta<MT, NW, META, kAGlobalPrep, L, DT>;
    case kALds: return k_rowmeta<MT, NW, META, kALds, L, DT>;
  }
  return nullptr;
}

template <int MT, int NW, int L, int DT>
DecodeKernel pick_mt_nw(const DecodePlan& p) {
  if (p.meta == kMetaGroup) return pick_ordered_spg<MT, NW, L, DT>(p.spg, p.amode, p.tn);
  if constexpr (NW <= 8 && !(MT == 4 && NW > 4)) {
    if (p.meta == kMetaRowLds) return pick_row_am<MT, NW, L, kMetaRowLds, DT>(p.amode);
    return pick_row_am<MT, NW, L, kMetaRowGlobal, DT>(p.amode);
  }
  return nullptr;
}

template <int MT, int L, int DT>
DecodeKernel pick_nw(const DecodePlan& p) {
  switch (p.nw) {
    case 4: return pick_mt_nw<MT, 4, L, DT>(p);
    case 8: return pick_mt_nw<MT, 8, L, DT>(p);
    case 16:
      if constexpr (MT < 4) return pick_mt_nw<MT, 16, L, DT>(p);
      return nullptr;
  }
  return nullptr;
}

template <int L, int DT>
DecodeKernel pick_layout(const DecodePlan& p) {
  switch (p.mt) {
    case 1: return pick_nw<1, L, DT>(p);
    case 2: return pick_nw<2, L, DT>(p);
    case 4: return pick_nw<4, L, DT>(p);
  }
  return nullptr;
}

template <int MT, int TN, bool PREP, int DT>
DecodeKernel pick_wide_spg(int spg) {
  switch (spg) {
    case 1: return k_wide<MT, kWideWaves, 1, TN, PREP, DT>;
    case 2: return k_wide<MT, kWideWaves, 2, TN, PREP, DT>;
    case 4: return k_wide<MT, kWideWaves, 4, TN, PREP, DT>;
    case 8: return k_wide<MT, kWideWaves, 8, TN, PREP, DT>;
  }
  return nullptr;
}

template <int DT>
DecodeKernel pick_wide(const DecodePlan& p) {
  const bool prep = p.amode == kAGlobalPrep;
  switch (p.mt) {
    case 1: return prep ? pick_wide_spg<1, 1, true, DT>(p.spg) : pick_wide_spg<1, 1, false, DT>(p.spg);
    case 2: return prep ? pick_wide_spg<2, 1, true, DT>(p.spg) : pick_wide_spg<2, 1, false, DT>(p.spg);
    case 4: return prep ? pick_wide_spg<4, 1, true, DT>(p.spg) : pick_wide_spg<4, 1, false, DT>(p.spg);
  }
  return nullptr;
}

// Gated kernels (silu(X W_gate) * (X W_up)): the ordered kernel with the
// two projections as its two weight streams (4 waves with X from global
// memory, 4 or 8 with X in LDS, as plan_decode gives), and the per-row kernel
// with a second stream. Instantiated in their own translation units.
template <int MT, int NW, int SPG, int L, int DT>
DecodeKernel pick_gated_ordered_am(int am) {
  switch (am) {
    case kAGlobal:
      if constexpr (NW == 4) return k_ordered<MT, NW, SPG, kAGlobal, L, 2, DT, true>;
      return nullptr;
    case kAGlobalPrep:
      if constexpr (NW == 4) return k_ordered<MT, NW, SPG, kAGlobalPrep, L, 2, DT, true>;
      return nullptr;
    case kALds: return k_ordered<MT, NW, SPG, kALds, L, 2, DT, true>;
    case kALdsGather: return k_ordered<MT, NW, SPG, kALdsGather, L, 2, DT, true>;
  }
  return nullptr;
}

template <int MT, int NW, int L, int DT>
DecodeKernel pick_gated_mt_nw(const DecodePlan& p) {
  if (p.meta == kMetaGroup) {
    switch (p.spg) {
      case 1: return pick_gated_ordered_am<MT, NW, 1, L, DT>(p.amode);
      case 2: return pick_gated_ordered_am<MT, NW, 2, L, DT>(p.amode);
      case 4: return pick_gated_ordered_am<MT, NW, 4, L, DT>(p.amode);
      case 8: return pick_gated_ordered_am<MT, NW, 8, L, DT>(p.amode);
    }
    return nullptr;
  }
  if constexpr (!(MT == 4 && NW > 4)) {
    const bool lds = p.meta == kMetaRowLds;
    switch (p.amode) {
      case kAGlobal:
        return lds ? k_rowmeta<MT, NW, kMetaRowLds, kAGlobal, L, DT, true>
                   : k_rowmeta<MT, NW, kMetaRowGlobal, kAGlobal, L, DT, true>;
      case kAGlobalPrep:
        return lds ? k_rowmeta<MT, NW, kMetaRowLds, kAGlobalPrep, L, DT, true>
                   : k_rowmeta<MT, NW, kMetaRowGlobal, kAGlobalPrep, L, DT, true>;
      case kALds:
        return lds ? k_rowmeta<MT, NW, kMetaRowLds, kALds, L, DT, true>
                   : k_rowmeta<MT, NW, kMetaRowGlobal, kALds, L, DT, true>;
    }
  }
  return nullptr;
}

template <int L, int DT>
DecodeKernel pick_gated_layout(const DecodePlan& p) {
  const int nw = p.nw;
  switch (p.mt) {
    case 1: return nw == 4 ? pick_gated_mt_nw<1, 4, L, DT>(p) : nw == 8 ? pick_gated_mt_nw<1, 8, L, DT>(p) : nullptr;
    case 2: return nw == 4 ? pick_gated_mt_nw<2, 4, L, DT>(p) : nullptr;  // 4 waves (plan_decode)
    case 4: return nw == 4 ? pick_gated_mt_nw<4, 4, L, DT>(p) : nullptr;
  }
  return nullptr;
}

template <int DT>
DecodeKernel pick_gated_dt(const DecodePlan& p) {
  if (p.layout == TPDQ_LAYOUT_TILED) return pick_gated_layout<TPDQ_LAYOUT_TILED, DT>(p);
  return pick_gated_layout<TPDQ_LAYOUT_GPTQ, DT>(p);
}

// the kernel of a plan: k_wide, or the tile kernel of its layout
template <int DT>
DecodeKernel pick_kernel_dt(const DecodePlan& p) {
  if (p.wide) return pick_wide<DT>(p);
  if (p.layout == TPDQ_LAYOUT_TILED) return pick_layout<TPDQ_LAYOUT_TILED, DT>(p);
  return pick_layout<TPDQ_LAYOUT_GPTQ, DT>(p);
}

}  // namespace
}  // namespace tpdq
