// Offline reorder on gfx950: Alg. 1 (P = argsort(g_idx), g_opt = g_idx[P])
// and the permutations of the packed weights and their metadata (section 2.2:
// W1[P1, P2], W2[P2]).
//
// The sort is a counting sort: with off[g] the number of rows in groups
// before g (an exclusive scan of the group counts, which the validation pass
// computes anyway), the sorted position of row i is
//   off[g_idx[i]] + #{ j < i : g_idx[j] == g_idx[i] }
// (ascending groups, ties by ascending row: the stable order). For Eq. 3's
// groups off[g] = g G. One workgroup per group sweeps g_idx in row order and
// ranks the group's members with wave ballots, so the result does not depend
// on scheduling.
#include "tpdq_internal.h"

namespace tpdq {
namespace {

__global__ void k_fill_u32(uint32_t* p, size_t n, uint32_t v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// flag bit 0: a g_idx value out of [0, num_groups); bit 1: a group whose
// count differs from what Eq. 3 gives (set by k_check_counts).
__global__ void k_count_groups(const int32_t* __restrict__ g_idx, int K, int num_groups,
                               uint32_t* __restrict__ counts, uint32_t* __restrict__ flag) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < K; i += gridDim.x * blockDim.x) {
    const uint32_t g = (uint32_t)g_idx[i];
    if (g >= (uint32_t)num_groups)
      atomicOr(flag, 1u);
    else
      atomicAdd(counts + g, 1u);
  }
}

// Eq. 3 with a permutation phi of 0..K-1: G rows in every group but the last,
// which holds K - (num_groups - 1) G (a partial group when G does not divide K)
__global__ void k_check_counts(const uint32_t* __restrict__ counts, int num_groups, int G, int K,
                               uint32_t* __restrict__ flag) {
  for (int g = blockIdx.x * blockDim.x + threadIdx.x; g < num_groups; g += gridDim.x * blockDim.x) {
    const uint32_t want = g == num_groups - 1 ? (uint32_t)(K - (num_groups - 1) * G) : (uint32_t)G;
    if (counts[g] != want) atomicOr(flag, 2u);
  }
}

// counts -> exclusive prefix sums, in place (one workgroup: 256 counts per
// pass into LDS, scanned serially there by thread 0, which carries the
// running total from pass to pass)
__global__ __launch_bounds__(256) void k_scan_counts(uint32_t* __restrict__ counts, int num_groups) {
  __shared__ uint32_t buf[256];
  uint32_t carry = 0;
  for (int c0 = 0; c0 < num_groups; c0 += 256) {
    const int g = c0 + (int)threadIdx.x;
    buf[threadIdx.x] = g < num_groups ? counts[g] : 0u;
    __syncthreads();
    if (threadIdx.x == 0) {
      for (int i = 0; i < 256; ++i) {
        const uint32_t v = buf[i];
        buf[i] = carry;
        carry += v;
      }
    }
    __syncthreads();
    if (g < num_groups) counts[g] = buf[threadIdx.x];
    __syncthreads();
  }
}

// One workgroup (256 threads = 4 waves) per group g; offs from k_scan_counts.
__global__ __launch_bounds__(256) void k_rank_group(const int32_t* __restrict__ g_idx, int K,
                                                    const uint32_t* __restrict__ offs, int num_groups,
                                                    int32_t* __restrict__ P,
                                                    int32_t* __restrict__ g_sorted) {
  __shared__ int wave_count[4];
  const int g = blockIdx.x;
  const int first = (int)offs[g];
  const int end = g + 1 < num_groups ? (int)offs[g + 1] : K;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int base = 0;  // members of group g already placed (rows before this chunk)
  for (int c0 = 0; c0 < K; c0 += 256) {
    const int i = c0 + threadIdx.x;
    const bool hit = i < K && g_idx[i] == g;
    const unsigned long long m = __ballot(hit);
    const int below = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wave_count[wave] = __popcll(m);
    __syncthreads();
    int before = base;
    for (int w = 0; w < wave; ++w) before += wave_count[w];
    const int total = wave_count[0] + wave_count[1] + wave_count[2] + wave_count[3];
    __syncthreads();
    if (hit) {
      const int r = first + before + below;
      if (r < end) {
        P[r] = i;
        g_sorted[r] = g;
      }
    }
    base += total;
  }
}

// One output word: rows P_row[8r .. 8r+7] of source column cs; nibble t of
// the result = nibble (i & 7) of src word [i >> 3][cs], i = P_row[8r + t].
__device__ __forceinline__ uint32_t gather_word(const uint32_t* __restrict__ src, int64_t ld_src,
                                                int K, const int32_t* __restrict__ Prow, int r,
                                                uint32_t cs) {
  if (!Prow) return src[(int64_t)r * ld_src + cs];
  const uint32_t kmax = (uint32_t)(K - 1);
  uint32_t out = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const uint32_t i = min((uint32_t)Prow[8 * r + t], kmax);
    const uint32_t w = src[(int64_t)(i >> 3) * ld_src + cs];
    out |= ((w >> (4 * (i & 7))) & 0xFu) << (4 * t);
  }
  return out;
}

// GPTQ-layout output: dst[r][c] = W[P_row, P_col] word.
__global__ void k_permute_qweight(const uint32_t* __restrict__ src, int64_t ld_src, int K, int N,
                                  const int32_t* __restrict__ Prow, const int32_t* __restrict__ Pcol,
                                  uint32_t* __restrict__ dst) {
  const int64_t words = (int64_t)(K / 8) * N;
  const uint32_t nmax = (uint32_t)(N - 1);
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < words;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(idx / N);
    const int c = (int)(idx - (int64_t)r * N);
    const uint32_t cs = Pcol ? min((uint32_t)Pcol[c], nmax) : (uint32_t)c;
    dst[idx] = gather_word(src, ld_src, K, Prow, r, cs);
  }
}

// A GPTQ word (row 8r + i at bits 4i) in the tiled nibble order: row 8r + i
// at bits 4 (i >> 1) + 16 (i & 1), the even rows in the low half-word and the
// odd rows in the high one.
__device__ __forceinline__ uint32_t interleave_nibbles(uint32_t w) {
  uint32_t out = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) out |= ((w >> (4 * i)) & 0xFu) << (4 * (i >> 1) + 16 * (i & 1));
  return out;
}

// Tiled output: dst[t][256 b + 4 l + u] = word [4 (4 b + u) + kq][16 t + j]
// with its nibbles interleaved, l = 16 kq + j; words past K or N are zero.
__global__ void k_permute_qweight_tiled(const uint32_t* __restrict__ src, int64_t ld_src, int K,
                                        int N, const int32_t* __restrict__ Prow,
                                        const int32_t* __restrict__ Pcol,
                                        uint32_t* __restrict__ dst) {
  const int64_t ld = tiled_ld(K);
  const int ntiles = (N + 15) / 16;
  const int64_t words = (int64_t)ntiles * ld;
  const uint32_t nmax = (uint32_t)(N - 1);
  const int kw = K / 8;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < words;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int t = (int)(idx / ld);
    const int o = (int)(idx - (int64_t)t * ld);
    const int b = o >> 8;
    const int l = (o >> 2) & 63;
    const int u = o & 3;
    const int r = 4 * (4 * b + u) + (l >> 4);
    const int c = 16 * t + (l & 15);
    uint32_t v = 0u;
    if (r < kw && c < N) {
      const uint32_t cs = Pcol ? min((uint32_t)Pcol[c], nmax) : (uint32_t)c;
      v = interleave_nibbles(gather_word(src, ld_src, K, Prow, r, cs));
    }
    dst[idx] = v;
  }
}

// dst[g][c] = src[g][P_col[c]] (2-byte elements; fp16 or bf16 bits).
__global__ void k_permute_scales(const uint16_t* __restrict__ src, int64_t ld_src, int ng, int N,
                                 const int32_t* __restrict__ Pcol, uint16_t* __restrict__ dst) {
  const int64_t total = (int64_t)ng * N;
  const uint32_t nmax = (uint32_t)(N - 1);
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int g = (int)(idx / N);
    const int c = (int)(idx - (int64_t)g * N);
    const uint32_t cs = Pcol ? min((uint32_t)Pcol[c], nmax) : (uint32_t)c;
    dst[idx] = src[(int64_t)g * ld_src + cs];
  }
}

// Zero codes packed along N: nibble t of dst word [g][cw] = zero of column
// P_col[8 cw + t] of group g.
__global__ void k_permute_qzeros(const uint32_t* __restrict__ src, int64_t ld_src, int ng, int N,
                                 const int32_t* __restrict__ Pcol, uint32_t* __restrict__ dst) {
  const int nw = N / 8;
  const int64_t total = (int64_t)ng * nw;
  const uint32_t nmax = (uint32_t)(N - 1);
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int g = (int)(idx / nw);
    const int cw = (int)(idx - (int64_t)g * nw);
    uint32_t out = 0;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t c = Pcol ? min((uint32_t)Pcol[8 * cw + t], nmax) : (uint32_t)(8 * cw + t);
      const uint32_t w = src[(int64_t)g * ld_src + (c >> 3)];
      out |= ((w >> (4 * (c & 7))) & 0xFu) << (4 * t);
    }
    dst[idx] = out;
  }
}

int grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 8192) b = 8192;
  if (b < 1) b = 1;
  return (int)b;
}

}  // namespace

hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t s) {
  hipLaunchKernelGGL(k_fill_u32, dim3(grid_for((int64_t)n)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_gidx_validate(const ReorderLayer& L, uint32_t* counts, uint32_t* flag,
                                hipStream_t s) {
  hipLaunchKernelGGL(k_count_groups, dim3(grid_for(L.K)), dim3(256), 0, s, L.g_idx, L.K,
                     L.num_groups, counts, flag);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || L.G == 0) return e;  // G == 0: groups of any size
  hipLaunchKernelGGL(k_check_counts, dim3(grid_for(L.num_groups)), dim3(256), 0, s, counts,
                     L.num_groups, L.G, L.K, flag);
  return hipGetLastError();
}

hipError_t launch_gidx_rank(const ReorderLayer& L, uint32_t* offs, hipStream_t s) {
  hipLaunchKernelGGL(k_scan_counts, dim3(1), dim3(256), 0, s, offs, L.num_groups);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rank_group, dim3(L.num_groups), dim3(256), 0, s, L.g_idx, L.K, offs,
                     L.num_groups, L.P, L.g_sorted);
  return hipGetLastError();
}

hipError_t launch_permute_qweight(const uint32_t* src, int64_t ld_src, int K, int N,
                                  const int32_t* Prow, const int32_t* Pcol, uint32_t* dst,
                                  int dst_layout, hipStream_t s) {
  if (dst_layout == TPDQ_LAYOUT_TILED) {
    const int64_t words = (int64_t)((N + 15) / 16) * tiled_ld(K);
    hipLaunchKernelGGL(k_permute_qweight_tiled, dim3(grid_for(words)), dim3(256), 0, s, src, ld_src,
                       K, N, Prow, Pcol, dst);
  } else {
    hipLaunchKernelGGL(k_permute_qweight, dim3(grid_for((int64_t)(K / 8) * N)), dim3(256), 0, s,
                       src, ld_src, K, N, Prow, Pcol, dst);
  }
  return hipGetLastError();
}

hipError_t launch_permute_scales(const uint16_t* src, int64_t ld_src, int ng, int N,
                                 const int32_t* Pcol, uint16_t* dst, hipStream_t s) {
  hipLaunchKernelGGL(k_permute_scales, dim3(grid_for((int64_t)ng * N)), dim3(256), 0, s, src,
                     ld_src, ng, N, Pcol, dst);
  return hipGetLastError();
}

hipError_t launch_permute_qzeros(const uint32_t* src, int64_t ld_src, int ng, int N,
                                 const int32_t* Pcol, uint32_t* dst, hipStream_t s) {
  hipLaunchKernelGGL(k_permute_qzeros, dim3(grid_for((int64_t)ng * (N / 8))), dim3(256), 0, s, src,
                     ld_src, ng, N, Pcol, dst);
  return hipGetLastError();
}

}  // namespace tpdq
