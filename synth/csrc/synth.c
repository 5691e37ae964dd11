/*
 * Seeded synthetic inputs for the OPT-shaped decoder workloads.
 *
 * This file draws random numbers and encodes them; it holds none of the
 * decoder's arithmetic.  Both the CPU oracle and the GPU library consume what
 * it writes (weights in fp16, or group-wise int4 codes of those fp16 values).
 *
 * Generator: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random
 * Numbers: As Easy as 1, 2, 3", SC'11), counter-based, so that any element
 * of any tensor can be regenerated on its own.  Element i of the stream
 * (key0, key1) comes from block b = i/8, whose counter is {b, 0, 0, 0}; its
 * four 64-bit outputs w[p] give one Box-Muller pair each (u1 from the low
 * 32 bits, u2 from the high 32 bits), producing elements 8b+2p (cosine
 * branch) and 8b+2p+1 (sine branch).
 *
 * fp16 encoding is IEEE binary16 with round-to-nearest-even (F16C).
 */
#include <immintrin.h>
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <omp.h>

typedef unsigned __int128 u128;

void synth_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    u128 p0 = (u128)0xD2E7470EE14C6C93ULL * c0;
    u128 p1 = (u128)0xCA5A826395121157ULL * c2;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    if (r < 9) { k0 += 0x9E3779B97F4A7C15ULL; k1 += 0xBB67AE8584CAA73BULL; }
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

uint16_t synth_f32_to_f16(float f) {
  return (uint16_t)_cvtss_sh(f, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC);
}

float synth_f16_to_f32(uint16_t h) { return _cvtsh_ss(h); }

/*
 * Sixty-four standard normals: blocks 8*grp .. 8*grp+7 of stream (key0, key1),
 * element e of the group being element 64*grp + e of the stream.  Computed in
 * fp32 (logf, sqrtf, sinf, cosf), always a whole group at a time, so a value
 * never depends on which range of the stream is requested.
 */
static void normal_group(uint64_t key0, uint64_t key1, uint64_t grp, float z[64]) {
  uint32_t ua[32], ub[32];
  const uint64_t key[2] = {key0, key1};
  for (int b = 0; b < 8; ++b) {
    const uint64_t ctr[4] = {grp * 8 + (uint64_t)b, 0, 0, 0};
    uint64_t w[4];
    synth_philox4x64_10(ctr, key, w);
    for (int p = 0; p < 4; ++p) {
      ua[b * 4 + p] = (uint32_t)w[p];
      ub[b * 4 + p] = (uint32_t)(w[p] >> 32);
    }
  }
  float r[32], th[32];
#pragma omp simd
  for (int i = 0; i < 32; ++i) {
    float u1 = ((float)(ua[i] >> 8) + 0.5f) * (1.0f / 16777216.0f); /* (0,1) */
    float u2 = (float)(ub[i] >> 8) * (1.0f / 16777216.0f);         /* [0,1) */
    r[i] = sqrtf(-2.0f * logf(u1));
    th[i] = 6.28318530717958647692f * u2;
  }
#pragma omp simd
  for (int i = 0; i < 32; ++i) {
    z[2 * i] = r[i] * cosf(th[i]);
    z[2 * i + 1] = r[i] * sinf(th[i]);
  }
}

/* out[j] = fp16(std * z[first + j]) (product in fp32), j in [0, n). */
void synth_normal_f16(uint64_t key0, uint64_t key1, uint64_t first, uint64_t n, double std,
                      uint16_t* out, int nthreads) {
  if (n == 0) return;
  const uint64_t g0 = first / 64, g1 = (first + n - 1) / 64;
  const float sd = (float)std;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
  for (int64_t grp = (int64_t)g0; grp <= (int64_t)g1; ++grp) {
    float z[64];
    normal_group(key0, key1, (uint64_t)grp, z);
    for (int e = 0; e < 64; ++e) {
      uint64_t i = (uint64_t)grp * 64 + (uint64_t)e;
      if (i < first || i >= first + n) continue;
      out[i - first] = synth_f32_to_f16(sd * z[e]);
    }
  }
}

/* out[j] = fp16(value) for all j (LayerNorm gamma = 1, beta = 0 and the like). */
void synth_fill_f16(uint16_t value_bits, uint64_t n, uint16_t* out) {
  for (uint64_t i = 0; i < n; ++i) out[i] = value_bits;
}

/*
 * Group-wise asymmetric int4 encoding of one fp16 row-major matrix W[N][K],
 * groups of 64 consecutive k inside a row.  Per group: mn, mx over the 64
 * values (as fp32); scale = (mx - mn) / 15; the stored pair is
 * {fp16(scale), fp16(mn)}; code = clamp(rint((w - min16) / scale16), 0, 15)
 * with ties to even (code 0 when scale16 == 0).  Codes are packed two per
 * byte, even k in the low nibble.  q is [N][K/2] bytes, sm is [N][K/64][2].
 */
static void quant_row(const uint16_t* w, int64_t K, uint8_t* q, uint16_t* sm) {
  for (int64_t g = 0; g < K / 64; ++g) {
    const uint16_t* wg = w + g * 64;
    float mn = INFINITY, mx = -INFINITY;
    for (int i = 0; i < 64; ++i) {
      float v = synth_f16_to_f32(wg[i]);
      mn = v < mn ? v : mn;
      mx = v > mx ? v : mx;
    }
    uint16_t s16 = synth_f32_to_f16((mx - mn) / 15.0f);
    uint16_t m16 = synth_f32_to_f16(mn);
    float s = synth_f16_to_f32(s16), m = synth_f16_to_f32(m16);
    sm[2 * g] = s16;
    sm[2 * g + 1] = m16;
    for (int i = 0; i < 64; i += 2) {
      int c[2];
      for (int e = 0; e < 2; ++e) {
        float v = synth_f16_to_f32(wg[i + e]);
        float r = s == 0.0f ? 0.0f : rintf((v - m) / s);
        c[e] = r < 0.0f ? 0 : (r > 15.0f ? 15 : (int)r);
      }
      q[(g * 64 + i) / 2] = (uint8_t)(c[0] | (c[1] << 4));
    }
  }
}

void synth_quant_int4_g64(const uint16_t* w, int64_t N, int64_t K, uint8_t* q, uint16_t* sm,
                          int nthreads) {
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
  for (int64_t n = 0; n < N; ++n) quant_row(w + n * K, K, q + n * (K / 2), sm + n * (K / 64) * 2);
}

/*
 * Draw W[N][K] = fp16(std * z) from stream (key0, key1) (element n*K + k) and
 * encode it as above without holding the fp16 matrix: the result equals
 * synth_quant_int4_g64 applied to synth_normal_f16's output.
 */
void synth_normal_int4_g64(uint64_t key0, uint64_t key1, int64_t N, int64_t K, double std,
                           uint8_t* q, uint16_t* sm, int nthreads) {
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : 1)
  {
    uint16_t row[65536 + 8];
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      for (int64_t k0 = 0; k0 < K; k0 += 65536) {
        int64_t len = K - k0 < 65536 ? K - k0 : 65536;
        synth_normal_f16(key0, key1, (uint64_t)(n * K + k0), (uint64_t)len, std, row, 1);
        quant_row(row, len, q + n * (K / 2) + k0 / 2, sm + (n * (K / 64) + k0 / 64) * 2);
      }
    }
  }
}
