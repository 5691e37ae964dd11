// Device-side helpers for gfx950 kernels (wave64, MFMA f16).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pipo {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float h2f(uint16_t h) {
  _Float16 v = __builtin_bit_cast(_Float16, h);
  return (float)v;
}
__device__ __forceinline__ uint16_t f2h(float f) {
  _Float16 v = (_Float16)f;  // round to nearest even
  return __builtin_bit_cast(uint16_t, v);
}

// 16-byte global load of 8 fp16 values
__device__ __forceinline__ h8 load_h8(const uint16_t* p) {
  return __builtin_bit_cast(h8, *reinterpret_cast<const u32x4*>(p));
}
// 16-byte loads of data read once per pass (streamed weights, KV-cache
// rows): non-temporal, so they do not displace reused lines from the caches
__device__ __forceinline__ u32x4 load_u32x4_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ h8 load_h8_stream(const uint16_t* p) {
  return __builtin_bit_cast(h8, load_u32x4_stream(p));
}
__device__ __forceinline__ h8 zero_h8() { return h8{0, 0, 0, 0, 0, 0, 0, 0}; }

// D = A . B + C for a 16x16 tile with K = 32 (v_mfma_f32_16x16x32_f16).
// Lane l supplies A[l % 16][8 * (l / 16) .. +8] and B[8 * (l / 16) .. +8][l % 16]
// (any permutation of k shared by A and B gives the same sum) and receives
// C[4 * (l / 16) + j][l % 16] in element j.
__device__ __forceinline__ f4 mfma16(h8 a, h8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// INT4 expansion.  A code c (0..15) placed in the low mantissa bits under
// the exponent of 1024.0 (fp16 0x6400, where the spacing is exactly 1) reads
// as 1024 + c; subtracting 1024 is exact, and one fused multiply-add gives
// c * s + m rounded once to fp16.  Two codes are expanded per packed fp16
// operation.  Codes come four bytes (eight codes, code 2i in the low nibble
// of byte i) to a 32-bit word.
typedef _Float16 h2 __attribute__((ext_vector_type(2)));

// (scale, min) pair word -> (s, s) and (m, m)
__device__ __forceinline__ void scale_min_pairs(uint32_t sm, h2& s2, h2& m2) {
  s2 = __builtin_bit_cast(h2, (sm & 0xFFFFu) | (sm << 16));
  m2 = __builtin_bit_cast(h2, (sm >> 16) | (sm & 0xFFFF0000u));
}

__device__ __forceinline__ h2 dequant_pair(uint32_t t, h2 s2, h2 m2) {
  const h2 c = __builtin_bit_cast(h2, t | 0x64006400u) - h2{(_Float16)1024.f, (_Float16)1024.f};
  return __builtin_elementwise_fma(c, s2, m2);
}

// eight codes in the order (0, 4, 1, 5, 2, 6, 3, 7).  Codes 0 and 4 (bits
// 0-3 and 16-19) go under the exponent of 1024 as above; codes 1 and 5
// (bits 4-7 and 20-23) are left where they are, under the exponent of 64
// (fp16 0x5400, spacing 1/16), where a code c at bits 4-7 reads as 64 + c:
// one AND-OR per pair and one shift per word, no per-pair shifts.  The
// biases 1024 and 64 are subtracted exactly before the fused multiply-add,
// so the values are those of dequant_pair.
__device__ __forceinline__ h2 dequant_biased(uint32_t t, _Float16 bias, h2 s2, h2 m2) {
  const h2 c = __builtin_bit_cast(h2, t) - h2{bias, bias};
  return __builtin_elementwise_fma(c, s2, m2);
}

// 32-bit constants the compiler sees as register values.  A three-operand
// instruction here encodes no literal and reads at most one scalar
// register, so (x & mask) | magic becomes a single v_and_or_b32 only with
// the mask in a scalar and the magic in a vector register.
__device__ __forceinline__ uint32_t sgpr_const(uint32_t v) {
  uint32_t r;
  asm("s_mov_b32 %0, %1" : "=s"(r) : "i"(v));
  return r;
}
__device__ __forceinline__ uint32_t vgpr_const(uint32_t v) {
  uint32_t r;
  asm("v_mov_b32 %0, %1" : "=v"(r) : "i"(v));
  return r;
}

__device__ __forceinline__ h8 dequant8_interleaved(uint32_t v, h2 s2, h2 m2) {
  const uint32_t v8 = v >> 8;
  const uint32_t e1024 = vgpr_const(0x64006400u), e64 = vgpr_const(0x54005400u);
  const uint32_t lo = sgpr_const(0x000F000Fu), hi = sgpr_const(0x00F000F0u);
  const h2 w0 = dequant_biased((v & lo) | e1024, (_Float16)1024.f, s2, m2);
  const h2 w1 = dequant_biased((v & hi) | e64, (_Float16)64.f, s2, m2);
  const h2 w2 = dequant_biased((v8 & lo) | e1024, (_Float16)1024.f, s2, m2);
  const h2 w3 = dequant_biased((v8 & hi) | e64, (_Float16)64.f, s2, m2);
  h8 out;
  out[0] = w0[0];
  out[1] = w0[1];
  out[2] = w1[0];
  out[3] = w1[1];
  out[4] = w2[0];
  out[5] = w2[1];
  out[6] = w3[0];
  out[7] = w3[1];
  return out;
}

// eight codes in natural order
__device__ __forceinline__ h8 dequant8(uint32_t v, h2 s2, h2 m2) {
  h8 out;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t b = v >> (8 * j);
    const h2 w = dequant_pair((b & 0xFu) | ((b << 12) & 0xF0000u), s2, m2);
    out[2 * j] = w[0];
    out[2 * j + 1] = w[1];
  }
  return out;
}

// eight fp16 values permuted to the order of dequant8_interleaved, so that
// an MFMA sees matching k on both operands
__device__ __forceinline__ h8 interleave_h8(h8 x) {
  const u32x4 d = __builtin_bit_cast(u32x4, x);
  u32x4 o;
  o[0] = (d[0] & 0xFFFFu) | (d[2] << 16);
  o[1] = (d[0] >> 16) | (d[2] & 0xFFFF0000u);
  o[2] = (d[1] & 0xFFFFu) | (d[3] << 16);
  o[3] = (d[1] >> 16) | (d[3] & 0xFFFF0000u);
  return __builtin_bit_cast(h8, o);
}

// Weight addressing, row-major or fragment order (PK).  In fragment order a
// 16-row x 32-k block of an fp16 matrix is 512 contiguous halves in MFMA
// operand order: lane slot L = r + 16 g (16 bytes) holds row r, k = 8 g ..
// 8 g + 7 of the block; blocks follow each other by k, then by row group,
// so the 64 lanes of a wave read 1 KiB contiguous per load.  INT4 codes:
// a 16-row x 128-k block is 1 KiB, lane slot r + 16 g holds row r's codes
// for k = 32 g .. 32 g + 31 (byte j: codes 2j, 2j+1 as in a row-major row);
// its (scale, min) pairs are 32 u32, row r's two groups at 2 r, 2 r + 1.
// Fragment order needs N % 16 == 0 (and K % 128 == 0 for INT4).
template <bool PK>
__device__ __forceinline__ int64_t w16_index(int64_t n, int64_t k, int64_t K) {
  if constexpr (PK)
    return ((n >> 4) * (K >> 5) + (k >> 5)) * 512 + (((n & 15) + 16 * ((k >> 3) & 3)) << 3) +
           (k & 7);
  else
    return n * K + k;
}
// byte of INT4 codes (k, k + 1), k even
template <bool PK>
__device__ __forceinline__ int64_t w4_byte(int64_t n, int64_t k, int64_t K) {
  if constexpr (PK)
    return ((n >> 4) * (K >> 7) + (k >> 7)) * 1024 + (((n & 15) + 16 * ((k >> 5) & 3)) << 4) +
           ((k & 31) >> 1);
  else
    return n * (K / 2) + k / 2;
}
// u32 index of the (scale, min) pair of the group holding k
template <bool PK>
__device__ __forceinline__ int64_t w4_sm(int64_t n, int64_t k, int64_t K) {
  if constexpr (PK)
    return ((n >> 4) * (K >> 7) + (k >> 7)) * 32 + (n & 15) * 2 + ((k >> 6) & 1);
  else
    return n * (K / 64) + k / 64;
}

// 16 bytes from global memory straight into LDS (global_load_lds_dwordx4):
// lane l of the wave writes bytes 16 l .. 16 l + 15 from `lds`, which must
// be the same for every lane.  Counted by vmcnt like any vector load.
__device__ __forceinline__ void lds_dma16(const void* g, uint8_t* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}
// s_waitcnt immediate: at most `vm` vector memory operations outstanding
// and, with lgkm0, no LDS operation (vmcnt bits 3:0 and 15:14, expcnt 6:4
// left at 7, lgkmcnt 11:8)
__device__ constexpr int waitcnt_imm(int vm, bool lgkm0) {
  return (vm & 15) | ((vm >> 4) << 14) | (7 << 4) | ((lgkm0 ? 0 : 15) << 8);
}

// Workgroup barrier without the fence of __syncthreads (whose release half
// waits for every outstanding vector load, prefetches into LDS included);
// the empty asm statements keep the compiler from moving memory operations
// across it.  LDS writes must have been waited for (s_waitcnt) before it.
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Transposed LDS read (ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane i receives element j (j = 0..3) from the 8-byte row that lane
// 4 j + i / 4 of the group addresses, at 16-bit position i % 4: the group's
// 16 addresses form a 4 x 16 matrix of halves and each lane gets a column.
typedef short s4 __attribute__((ext_vector_type(4)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ h4 lds_read_tr16(const uint8_t* lds) {
  // the whole vector is reinterpreted: clang's bit_cast of a single vector
  // element reads element 0
  return __builtin_bit_cast(
      h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)lds));
}

template <typename T>
__device__ __forceinline__ T wave_shfl_xor(T v, int mask) {
  return __shfl_xor(v, mask, 64);
}

}  // namespace pipo
