// Causal softmax attention over a position-major KV cache: row p * b + i
// of K (or V) holds sequence i's key (value) at position p, all heads side
// by side.  This is the layout the copy engine streams when the cache lives
// in host memory: a layer's prefix 0..t-1 is one contiguous range.
//
//   attn_decode:  one new query per (sequence, head) against keys 0..t.
//   attn_prefill: P queries per (sequence, head), causal, flash-style with
//                 v_mfma_f32_16x16x32_f16 for Q K^T and P V.
// Softmax is max-subtracted in fp32; every reduction has a fixed order.
#include <cfloat>

#include "common.h"
#include "device.h"

namespace pipo {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// ---------------------------------------------------------------------------
// decode: grid (heads, b), 256 threads.  A position is handled by D/8 lanes
// (8 dims each); scores for all t+1 keys are held in LDS, then normalised,
// then V is accumulated.  K and V rows are read once, 16 bytes per lane.
template <int D>
__global__ __launch_bounds__(256) void attn_decode_k(const uint16_t* __restrict__ q,
                                                     const uint16_t* __restrict__ kc,
                                                     const uint16_t* __restrict__ vc,
                                                     uint16_t* __restrict__ o, int b, int H,
                                                     int t) {
  extern __shared__ float sc[];  // [t + 1]
  __shared__ float part[4][D];
  __shared__ float red[4];
  constexpr int LPP = D / 8;     // lanes per position
  constexpr int PPW = 64 / LPP;  // positions per wave per pass
  const int h = blockIdx.x, bi = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane / LPP, cl = lane % LPP;
  const int64_t d = (int64_t)H * D;
  const int T = t + 1;
  const int64_t col = (int64_t)h * D + cl * 8;

  float qf[8];
  {
    const h8 qv = load_h8(q + (int64_t)bi * d + col);
#pragma unroll
    for (int i = 0; i < 8; ++i) qf[i] = (float)qv[i];
  }
  for (int p = wave * PPW + sub; p < T; p += 4 * PPW) {
    const h8 kv = load_h8(kc + ((int64_t)p * b + bi) * d + col);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += qf[i] * (float)kv[i];
#pragma unroll
    for (int off = LPP / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    if (cl == 0) sc[p] = s;
  }
  __syncthreads();

  float mx = -FLT_MAX;
  for (int p = tid; p < T; p += 256) mx = fmaxf(mx, sc[p]);
  mx = wave_max(mx);
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sum = 0.f;
  for (int p = tid; p < T; p += 256) {
    const float e = expf(sc[p] - mx);
    sc[p] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  if (lane == 0) red[wave] = sum;
  __syncthreads();
  sum = red[0] + red[1] + red[2] + red[3];

  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int p = wave * PPW + sub; p < T; p += 4 * PPW) {
    const h8 vv = load_h8(vc + ((int64_t)p * b + bi) * d + col);
    const float w = sc[p];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += w * (float)vv[i];
  }
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int off = LPP; off < 64; off <<= 1) acc[i] += __shfl_xor(acc[i], off, 64);
  if (sub == 0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) part[wave][cl * 8 + i] = acc[i];
  }
  __syncthreads();
  const float inv = 1.f / sum;
  for (int c = tid; c < D; c += 256) {
    const float v = ((part[0][c] + part[1][c]) + part[2][c]) + part[3][c];
    o[(int64_t)bi * d + (int64_t)h * D + c] = f2h(v * inv);
  }
}

// ---------------------------------------------------------------------------
// prefill: grid (ceil(P / 64), heads, b), 4 waves x 16 queries.  Keys come
// in blocks of 64 (K row-major and V transposed in LDS); each wave keeps an
// online softmax per query row and its O tile in MFMA accumulators.
template <int D>
__global__ __launch_bounds__(256) void attn_prefill_k(const uint16_t* __restrict__ q,
                                                      const uint16_t* __restrict__ kc,
                                                      const uint16_t* __restrict__ vc,
                                                      uint16_t* __restrict__ o, int b, int P,
                                                      int H) {
  constexpr int KB = 64;
  constexpr int KROW = D + 8;
  constexpr int VROW = KB + 8;
  constexpr int PROW = KB + 8;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KB * KROW];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VROW];
  __shared__ __attribute__((aligned(16))) uint16_t Ps[4][16 * PROW];

  const int qb = blockIdx.x, h = blockIdx.y, bi = blockIdx.z;
  const int64_t d = (int64_t)H * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int q0 = qb * 64 + wave * 16;

  h8 qf[D / 32];
  {
    const int qp = q0 + r;
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk)
      qf[kk] = qp < P ? load_h8(q + ((int64_t)bi * P + qp) * d + (int64_t)h * D + 32 * kk + 8 * g)
                      : zero_h8();
  }
  f4 oacc[D / 16];
#pragma unroll
  for (int n = 0; n < D / 16; ++n) oacc[n] = f4{0.f, 0.f, 0.f, 0.f};
  float mrow[4], lrow[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    mrow[e] = -INFINITY;
    lrow[e] = 0.f;
  }

  for (int kb = 0; kb <= qb; ++kb) {
    __syncthreads();
    for (int c = tid; c < KB * (D / 8); c += 256) {
      const int key = c / (D / 8), col = (c % (D / 8)) * 8;
      const int kp = kb * KB + key;
      const int64_t off = ((int64_t)kp * b + bi) * d + (int64_t)h * D + col;
      const h8 kv = kp < P ? load_h8(kc + off) : zero_h8();
      const h8 vv = kp < P ? load_h8(vc + off) : zero_h8();
      *reinterpret_cast<h8*>(&Ks[key * KROW + col]) = kv;
      const u32x4 vw = __builtin_bit_cast(u32x4, vv);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        Vt[(col + i) * VROW + key] = (uint16_t)(vw[i >> 1] >> (16 * (i & 1)));
    }
    __syncthreads();

    f4 s[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      s[j] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) {
        const h8 kf = *reinterpret_cast<const h8*>(&Ks[(j * 16 + r) * KROW + 32 * kk + 8 * g]);
        s[j] = mfma16(qf[kk], kf, s[j]);
      }
    }
    // s[j][e]: query q0 + 4 g + e, key kb * 64 + 16 j + r
    float bm[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int qpos = q0 + 4 * g + e;
      bm[e] = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = kb * KB + 16 * j + r;
        if (key > qpos || key >= P) s[j][e] = -INFINITY;
        bm[e] = fmaxf(bm[e], s[j][e]);
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) bm[e] = fmaxf(bm[e], __shfl_xor(bm[e], off, 64));
    }
    float alpha[4], rs[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float mnew = fmaxf(mrow[e], bm[e]);
      alpha[e] = mrow[e] == -INFINITY ? 0.f : expf(mrow[e] - mnew);
      mrow[e] = mnew;
      rs[e] = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p = expf(s[j][e] - mnew);
        s[j][e] = p;
        rs[e] += p;
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) rs[e] += __shfl_xor(rs[e], off, 64);
      lrow[e] = lrow[e] * alpha[e] + rs[e];
    }
#pragma unroll
    for (int n = 0; n < D / 16; ++n)
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[n][e] *= alpha[e];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) Ps[wave][(4 * g + e) * PROW + 16 * j + r] = f2h(s[j][e]);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KB / 32; ++kk) {
      const h8 pf = *reinterpret_cast<const h8*>(&Ps[wave][r * PROW + 32 * kk + 8 * g]);
#pragma unroll
      for (int n = 0; n < D / 16; ++n) {
        const h8 vf = *reinterpret_cast<const h8*>(&Vt[(16 * n + r) * VROW + 32 * kk + 8 * g]);
        oacc[n] = mfma16(pf, vf, oacc[n]);
      }
    }
  }

#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int qpos = q0 + 4 * g + e;
    if (qpos >= P) continue;
    const float inv = 1.f / lrow[e];
    uint16_t* orow = o + ((int64_t)bi * P + qpos) * d + (int64_t)h * D;
#pragma unroll
    for (int n = 0; n < D / 16; ++n) orow[16 * n + r] = f2h(oacc[n][e] * inv);
  }
}

// ---------------------------------------------------------------------------
pipo_status launch_attn_decode(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                               uint16_t* o, int b, int n_heads, int head_dim, int t,
                               hipStream_t st) {
  if (b < 1 || n_heads < 1 || t < 0) {
    set_error("attn_decode: bad shape b=%d heads=%d t=%d", b, n_heads, t);
    return PIPO_ERR_ARG;
  }
  if (t + 1 > kAttnDecodeMaxT) {
    set_error("attn_decode: %d keys exceed the %d the kernel holds", t + 1, kAttnDecodeMaxT);
    return PIPO_ERR_UNSUPPORTED;
  }
  const dim3 grid((unsigned)n_heads, (unsigned)b);
  const size_t lds = (size_t)(t + 1) * sizeof(float);
  if (head_dim == 128) {
    hipLaunchKernelGGL(attn_decode_k<128>, grid, dim3(256), lds, st, q, kc, vc, o, b, n_heads, t);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL(attn_decode_k<64>, grid, dim3(256), lds, st, q, kc, vc, o, b, n_heads, t);
  } else {
    set_error("attn_decode: head_dim %d not supported (64 or 128)", head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_attn_prefill(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                uint16_t* o, int b, int P, int n_heads, int head_dim,
                                hipStream_t st) {
  if (b < 1 || n_heads < 1 || P < 1) {
    set_error("attn_prefill: bad shape b=%d P=%d heads=%d", b, P, n_heads);
    return PIPO_ERR_ARG;
  }
  const dim3 grid((unsigned)((P + 63) / 64), (unsigned)n_heads, (unsigned)b);
  if (head_dim == 128) {
    hipLaunchKernelGGL(attn_prefill_k<128>, grid, dim3(256), 0, st, q, kc, vc, o, b, P, n_heads);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL(attn_prefill_k<64>, grid, dim3(256), 0, st, q, kc, vc, o, b, P, n_heads);
  } else {
    set_error("attn_prefill: head_dim %d not supported (64 or 128)", head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

}  // namespace pipo
