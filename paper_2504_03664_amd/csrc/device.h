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
__device__ __forceinline__ h8 zero_h8() { return h8{0, 0, 0, 0, 0, 0, 0, 0}; }

// D = A . B + C for a 16x16 tile with K = 32 (v_mfma_f32_16x16x32_f16).
// Lane l supplies A[l % 16][8 * (l / 16) .. +8] and B[8 * (l / 16) .. +8][l % 16]
// (any permutation of k shared by A and B gives the same sum) and receives
// C[4 * (l / 16) + j][l % 16] in element j.
__device__ __forceinline__ f4 mfma16(h8 a, h8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// expand 32 int4 codes (16 bytes, code 2i in the low nibble of byte i) to
// fp16 (code * s + m, computed in fp32) as four groups of eight
__device__ __forceinline__ void dequant32(u32x4 codes, float s, float m, h8 out[4]) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t v = codes[w];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float c = (float)((v >> (4 * i)) & 0xFu);
      out[w][i] = (_Float16)__builtin_fmaf(c, s, m);
    }
  }
}

template <typename T>
__device__ __forceinline__ T wave_shfl_xor(T v, int mask) {
  return __shfl_xor(v, mask, 64);
}

}  // namespace pipo
