// Device helpers shared by the GEMM kernels of libtpdq (gfx950): fp16 and
// bf16 vector types, the exact int4 unpack, MFMA and wait-count wrappers, and
// raw buffer loads. Included by the .hip translation units only.
#pragma once

#include "tpdq_internal.h"

namespace tpdq {
namespace {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef __bf16 b2_t __attribute__((ext_vector_type(2)));
typedef __bf16 b8_t __attribute__((ext_vector_type(8)));
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

// Element type of activations, scales and outputs (tpdq_dtype).
constexpr int kF16 = TPDQ_FP16;
constexpr int kBF16 = TPDQ_BF16;

template <int DT>
__device__ __forceinline__ float bits_to_float(uint32_t bits16) {
  if constexpr (DT == kBF16) return as_f32(bits16 << 16);  // bf16 is the top half of an fp32
  else return half_bits_to_float(bits16);
}

template <int DT>
__device__ __forceinline__ uint16_t float_to_bits(float f) {
  if constexpr (DT == kBF16) return __builtin_bit_cast(uint16_t, (__bf16)f);  // nearest even
  else return float_to_half_bits(f);
}

// {a, b} rounded to the element type, a in the low half-word
template <int DT>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  if constexpr (DT == kBF16) {
    const b2_t v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v);
  } else {
    const h2_t v = {(_Float16)a, (_Float16)b};
    return as_u32(v);
  }
}

// Packed word -> 8 fp16 values (q - z) of one column, exact.
// OR-ing a nibble into the mantissa of 1024.0 (0x6400) gives 1024 + q; the
// nibbles at bits 4..7 land as 1024 + 16 q and are rescaled by 1/16 inside
// the same fused op. The value pairs come from nibble positions (0, 4),
// (1, 5), (2, 6), (3, 7): for a GPTQ word (row 8r + i at position i) that is
// rows k0, k4, k1, k5, k2, k6, k3, k7, and the A operand is permuted to match
// (permute_octet); a tiled word stores row 8r + i at position
// 4 (i >> 1) + 16 (i & 1) (even rows in the low half-word, odd rows in the
// high one), so the values come out as k0 .. k7 and A is used as loaded.
// The masks live in VGPRs (v_and_or_b32 takes no two literals and reads one
// SGPR at most on this ISA), so each pair costs one v_and_or_b32.
// For bf16 the magic number is 128.0 (0x4300): 128 + q is exact (bf16 holds
// the integers 128 .. 255), and the zero is not subtracted per element (see
// unpack_bias_bf16).
template <int DT = kF16>
struct UnpackConsts {
  uint32_t lo, hi, magic;
  __device__ __forceinline__ UnpackConsts() {
    asm volatile("v_mov_b32 %0, 0x000f000f" : "=v"(lo));
    asm volatile("v_mov_b32 %0, 0x00f000f0" : "=v"(hi));
    if constexpr (DT == kBF16)
      asm volatile("v_mov_b32 %0, 0x43004300" : "=v"(magic));
    else
      asm volatile("v_mov_b32 %0, 0x64006400" : "=v"(magic));
  }
};

__device__ __forceinline__ h8_t unpack_sub(const UnpackConsts<kF16>& k, uint32_t w, uint32_t z1024,
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

// Packed word -> 8 bf16 values 128 + q of one column, exact, in the order of
// unpack_sub (nibble positions (0, 4), (1, 5), (2, 6), (3, 7)). bf16 has no
// packed arithmetic here to subtract the zero per element, so the zero is
// applied once per group instead: sum_k x (q - z) = sum_k x (128 + q) -
// (128 + z) sum_k x, with sum_k x taken by the same MFMA against ones.
__device__ __forceinline__ u4_t unpack_bias_bf16(const UnpackConsts<kBF16>& k, uint32_t w) {
  const uint32_t lo = k.lo, magic = k.magic;
  u4_t r;
  r.x = (w & lo) | magic;
  r.y = ((w >> 4) & lo) | magic;
  r.z = ((w >> 8) & lo) | magic;
  r.w = ((w >> 12) & lo) | magic;
  return r;
}

// bf16 ones: the B operand whose product with A sums A's 32 columns
constexpr uint32_t kBf16OnePair = 0x3F803F80u;

// The B operand of one 32-row step: fp16 q - z (the zero subtracted per
// element), or bf16 128 + q (the zero applied per group).
template <int DT>
__device__ __forceinline__ u4_t unpack_step(const UnpackConsts<DT>& k, uint32_t w, uint32_t z1024,
                                            uint32_t z64) {
  if constexpr (DT == kBF16) return unpack_bias_bf16(k, w);
  else return __builtin_bit_cast(u4_t, unpack_sub(k, w, z1024, z64));
}


// Per-row dequant of one word: row r (0..7) has zero z[r] and scale bits
// s[r]; returns fp16(s * (q - z)) in the unpack order of the word's layout
// (NAT: a tiled word, rows k0 .. k7; else k0, k4, k1, k5, k2, k6, k3, k7).
template <bool NAT>
__device__ __forceinline__ h8_t dequant_rows_f16(const UnpackConsts<kF16>& k, uint32_t w,
                                                 const uint32_t (&z)[8], const uint32_t (&s)[8]) {
  const uint32_t lo = k.lo, hi = k.hi, magic = k.magic;
  const uint32_t w8 = w >> 8;
  const h2_t inv16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  // rows held by nibble positions 0, 1, 2, 3 (low halves) and 4, 5, 6, 7
  constexpr int r0 = 0, r1 = NAT ? 2 : 1, r2 = NAT ? 4 : 2, r3 = NAT ? 6 : 3;
  constexpr int r4 = NAT ? 1 : 4, r5 = NAT ? 3 : 5, r6 = NAT ? 5 : 6, r7 = 7;
  const uint32_t z04 = ((0x6400u | z[r0]) | ((0x6400u | z[r4]) << 16));
  const uint32_t z15 = ((0x5400u | (z[r1] << 4)) | ((0x5400u | (z[r5] << 4)) << 16));
  const uint32_t z26 = ((0x6400u | z[r2]) | ((0x6400u | z[r6]) << 16));
  const uint32_t z37 = ((0x5400u | (z[r3] << 4)) | ((0x5400u | (z[r7] << 4)) << 16));
  u4_t r;
  r.x = as_u32((as_h2((w & lo) | magic) - as_h2(z04)) * as_h2(s[r0] | (s[r4] << 16)));
  r.y = as_u32((as_h2((w & hi) | magic) * inv16 - as_h2(z15)) * as_h2(s[r1] | (s[r5] << 16)));
  r.z = as_u32((as_h2((w8 & lo) | magic) - as_h2(z26)) * as_h2(s[r2] | (s[r6] << 16)));
  r.w = as_u32((as_h2((w8 & hi) | magic) * inv16 - as_h2(z37)) * as_h2(s[r3] | (s[r7] << 16)));
  return as_h8(r);
}

// The same for bf16: s * (q - z) formed in fp32 (exact: an 8-bit scale times
// a small integer) and rounded once to bf16.
template <bool NAT, int DT>
__device__ __forceinline__ u4_t dequant_rows(const UnpackConsts<DT>& k, uint32_t w,
                                             const uint32_t (&z)[8], const uint32_t (&s)[8]) {
  if constexpr (DT == kF16) {
    return __builtin_bit_cast(u4_t, dequant_rows_f16<NAT>(k, w, z, s));
  } else {
    // nibble position p holds row p (GPTQ) or row 2p, 2 (p - 4) + 1 (tiled)
    auto val = [&](int p) {
      const int r = NAT ? (p < 4 ? 2 * p : 2 * (p - 4) + 1) : p;
      const int q = (int)((w >> (4 * p)) & 0xFu);
      return (float)(q - (int)z[r]) * bits_to_float<kBF16>(s[r]);
    };
    u4_t out;
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = pack2<kBF16>(val(i), val(i + 4));
    return out;
  }
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

// Activations as loaded -> the A operand for weights of the given layout.
template <int LAYOUT>
__device__ __forceinline__ u4_t to_operand(u4_t x) {
  if constexpr (LAYOUT == TPDQ_LAYOUT_TILED) return x;
  else return permute_octet(x);
}

// s_waitcnt vmcnt(N) alone (expcnt and lgkmcnt at their maxima). Placed
// where the N most recent vector-memory loads may stay in flight while all
// older ones must have landed; it also tells the compiler's wait-count pass
// that the older loads are done on every path.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ f4_t mfma16x16x32(h8_t a, h8_t b, f4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_{f16,bf16} on raw operand bits
template <int DT>
__device__ __forceinline__ f4_t mfma_k32(u4_t a, u4_t b, f4_t c) {
  if constexpr (DT == kBF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8_t, a),
                                                   __builtin_bit_cast(b8_t, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(a), as_h8(b), c, 0, 0, 0);
}

// Workgroups are dispatched round-robin over the 8 XCDs. Neighbouring
// 16-column tiles share 128-byte lines of scales (and, in the GPTQ layout, of
// qweight), so consecutive tiles go to workgroups on the same XCD (same L2).
__device__ __forceinline__ int xcd_tile(int b, int nb) {
  if (nb % 8) return b;
  return (b % 8) * (nb / 8) + b / 8;
}

// Buffer loads. A raw buffer resource carries its size: a load past it
// returns zeros without touching memory. Loads therefore need no branches
// (every item, valid or not, issues exactly one load, which keeps the wait
// counts exact), and items past the data cost no traffic.
constexpr uint32_t kOutOfRange = 0x80000000u;  // an offset past every resource here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  // stride 0 (raw), 32-bit dwords, range checked against `bytes`
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}
// kNonTemporal: the cache-policy bit for data read once (the weight stream)
constexpr int kNonTemporal = 2;
template <int POLICY = 0>
__device__ __forceinline__ u4_t buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, POLICY));
}
template <int POLICY = 0>
__device__ __forceinline__ uint32_t buffer_load4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, POLICY);
}

__device__ __forceinline__ uint32_t buffer_load2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}

}  // namespace
}  // namespace tpdq
