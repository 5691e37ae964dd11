// INT4 KV cache rows (Section 2: the KV cache may be kept in 4 bits; the
// conversion belongs to the cache's loading and saving, Section 3.1.2).
// A row of d elements: d/2 code bytes, element 2i in the low nibble of byte
// i, then d/64 fp16 (scale, min) pairs, one per 64 consecutive elements.
//
//   kv_quant_k:   fp16 rows -> INT4 rows; per group, in fp32:
//                 scale = fp16((max - min) / 15), min = fp16(min),
//                 code = clamp(rint((x - min) / scale), 0, 15), half to
//                 even, 0 where scale is 0 (both divisions IEEE-rounded).
//   kv_dequant_k: INT4 rows -> fp16 rows, code * scale + min rounded once.
// One thread per group of 64: 128 bytes in, 36 out (or the reverse).
#include "common.h"
#include "device.h"

namespace pipo {

__global__ __launch_bounds__(256) void kv_quant_k(const uint16_t* __restrict__ x,
                                                  uint8_t* __restrict__ out, int64_t rows,
                                                  int64_t d) {
  const int64_t groups = d / 64;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= rows * groups) return;
  const int64_t r = e / groups, gi = e % groups;
  const uint16_t* src = x + r * d + gi * 64;
  float v[64];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const h8 h = load_h8(src + 8 * i);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[8 * i + j] = (float)h[j];
  }
  float mn = v[0], mx = v[0];
#pragma unroll
  for (int i = 1; i < 64; ++i) {
    mn = fminf(mn, v[i]);
    mx = fmaxf(mx, v[i]);
  }
  const _Float16 s16 = (_Float16)((mx - mn) / 15.f);
  const _Float16 m16 = (_Float16)mn;
  const float s = (float)s16, m = (float)m16;
  u32x4 codes[2];
#pragma unroll
  for (int w = 0; w < 8; ++w) {
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float c = 0.f;
      if (s != 0.f) c = fminf(fmaxf(__builtin_rintf((v[8 * w + j] - m) / s), 0.f), 15.f);
      word |= (uint32_t)c << (4 * j);
    }
    codes[w >> 2][w & 3] = word;
  }
  uint8_t* row = out + r * (d / 2 + d / 16);
  *reinterpret_cast<u32x4*>(row + gi * 32) = codes[0];
  *reinterpret_cast<u32x4*>(row + gi * 32 + 16) = codes[1];
  *reinterpret_cast<uint32_t*>(row + d / 2 + gi * 4) =
      (uint32_t)__builtin_bit_cast(uint16_t, s16) | ((uint32_t)__builtin_bit_cast(uint16_t, m16) << 16);
}

__global__ __launch_bounds__(256) void kv_dequant_k(const uint8_t* __restrict__ in,
                                                    uint16_t* __restrict__ y, int64_t rows,
                                                    int64_t d) {
  const int64_t groups = d / 64;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= rows * groups) return;
  const int64_t r = e / groups, gi = e % groups;
  const uint8_t* row = in + r * (d / 2 + d / 16);
  const u32x4 c0 = *reinterpret_cast<const u32x4*>(row + gi * 32);
  const u32x4 c1 = *reinterpret_cast<const u32x4*>(row + gi * 32 + 16);
  h2 s2, m2;
  scale_min_pairs(*reinterpret_cast<const uint32_t*>(row + d / 2 + gi * 4), s2, m2);
  uint16_t* dst = y + r * d + gi * 64;
#pragma unroll
  for (int w = 0; w < 8; ++w) {
    const h8 h = dequant8(w < 4 ? c0[w] : c1[w - 4], s2, m2);
    *reinterpret_cast<h8*>(dst + 8 * w) = h;
  }
}

pipo_status launch_kv_quant(const uint16_t* x, uint8_t* out, int64_t rows, int64_t d,
                            hipStream_t st) {
  if (rows < 0 || d <= 0 || d % 256 != 0) {
    set_error("kv_quant: rows %lld, d %lld (d must be a multiple of 256)", (long long)rows,
              (long long)d);
    return PIPO_ERR_UNSUPPORTED;
  }
  const int64_t n = rows * (d / 64);
  if (n == 0) return PIPO_OK;
  launch(kv_quant_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, x, out, rows, d);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_kv_dequant(const uint8_t* in, uint16_t* y, int64_t rows, int64_t d,
                              hipStream_t st) {
  if (rows < 0 || d <= 0 || d % 256 != 0) {
    set_error("kv_dequant: rows %lld, d %lld (d must be a multiple of 256)", (long long)rows,
              (long long)d);
    return PIPO_ERR_UNSUPPORTED;
  }
  const int64_t n = rows * (d / 64);
  if (n == 0) return PIPO_OK;
  launch(kv_dequant_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, in, y, rows, d);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

}  // namespace pipo
