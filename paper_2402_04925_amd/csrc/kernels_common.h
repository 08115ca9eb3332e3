// Device helpers shared by the GEMM kernels of libtpdq (gfx950): fp16
// vector types, the exact int4 unpack, MFMA and wait-count wrappers, and
// raw buffer loads. Included by the .hip translation units only.
#pragma once

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
// the same fused op. The value pairs come from nibble positions (0, 4),
// (1, 5), (2, 6), (3, 7): for a GPTQ word (row 8r + i at position i) that is
// rows k0, k4, k1, k5, k2, k6, k3, k7, and the A operand is permuted to match
// (permute_octet); a tiled word stores row 8r + i at position
// 4 (i >> 1) + 16 (i & 1) (even rows in the low half-word, odd rows in the
// high one), so the values come out as k0 .. k7 and A is used as loaded.
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
// s[r]; returns fp16(s * (q - z)) in the unpack order of the word's layout
// (NAT: a tiled word, rows k0 .. k7; else k0, k4, k1, k5, k2, k6, k3, k7).
template <bool NAT>
__device__ __forceinline__ h8_t dequant_rows(const UnpackConsts& k, uint32_t w,
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
