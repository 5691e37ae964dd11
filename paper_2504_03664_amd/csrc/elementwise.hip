// Row-wise kernels of the decoder: LayerNorm and RMSNorm, embedding, rotary
// positions, the SwiGLU gate, greedy argmax, and a fill used to poison
// weight slots.  The residual stream x is fp32; the normalised output that
// feeds the next GEMM is fp16.
#include <cfloat>
#include <climits>

#include "common.h"
#include "device.h"

namespace pipo {

typedef float f4v __attribute__((ext_vector_type(4)));

// sum over a 256-thread block in a fixed order (waves, then wave 0..3)
__device__ __forceinline__ float block_sum256(float v, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

// LayerNorm: y[r] = (x[src] - mean) / sqrt(var + eps) * gamma + beta, two
// passes over the row held in registers (d <= 256 * 4 * kLnMaxVec).
// RMSNorm (RMS): y[r] = x[src] / sqrt(mean(x^2) + eps) * gamma.
constexpr int kLnMaxVec = 8;

template <bool RMS>
__global__ __launch_bounds__(256) void norm_k(const float* __restrict__ x,
                                                   const uint16_t* __restrict__ gamma,
                                                   const uint16_t* __restrict__ beta,
                                                   uint16_t* __restrict__ y, int64_t d,
                                                   int64_t src_stride, int64_t src_offset,
                                                   float eps) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const f4v* xr = reinterpret_cast<const f4v*>(x + (row * src_stride + src_offset) * d);
  const int nv = (int)(d / 4);
  const int tid = threadIdx.x;
  f4v v[kLnMaxVec];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kLnMaxVec; ++i) {
    const int c = tid + 256 * i;
    v[i] = c < nv ? xr[c] : f4v{0.f, 0.f, 0.f, 0.f};
    s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
  }
  const float mean = RMS ? 0.f : block_sum256(s, red) / (float)d;
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < kLnMaxVec; ++i) {
    const int c = tid + 256 * i;
    if (c < nv) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t = v[i][e] - mean;
        sq += t * t;
      }
    }
  }
  const float var = block_sum256(sq, red) / (float)d;
  const float rstd = 1.f / sqrtf(var + eps);
  uint16_t* yr = y + row * d;
#pragma unroll
  for (int i = 0; i < kLnMaxVec; ++i) {
    const int c = tid + 256 * i;
    if (c < nv) {
      u32x2 packed;
#pragma unroll
      for (int e = 0; e < 4; e += 2) {
        const int64_t k = 4 * (int64_t)c + e;
        float a0 = (v[i][e] - mean) * rstd * h2f(gamma[k]);
        float a1 = (v[i][e + 1] - mean) * rstd * h2f(gamma[k + 1]);
        if constexpr (!RMS) {
          a0 += h2f(beta[k]);
          a1 += h2f(beta[k + 1]);
        }
        packed[e / 2] = (uint32_t)f2h(a0) | ((uint32_t)f2h(a1) << 16);
      }
      *reinterpret_cast<u32x2*>(yr + 4 * (int64_t)c) = packed;
    }
  }
}

// x[r][:] = tok(r) + pos_table[pos0 + r % rows_per_seq + pos_offset], with
// tok(r) = tok_rows[r] (gathered on the host) or tok_table[ids[r]]; without
// a position table x[r][:] = tok(r)
__global__ __launch_bounds__(256) void embed_k(const uint16_t* __restrict__ tok_rows,
                                               const int32_t* __restrict__ ids,
                                               const uint16_t* __restrict__ tok_table,
                                               const uint16_t* __restrict__ pos_table,
                                               float* __restrict__ x, int64_t d,
                                               int64_t rows_per_seq, int64_t pos0,
                                               int64_t pos_offset) {
  const int64_t r = blockIdx.x;
  const uint16_t* tr = tok_rows ? tok_rows + r * d : tok_table + (int64_t)ids[r] * d;
  if (!pos_table) {
    for (int64_t c = threadIdx.x; c < d; c += 256) x[r * d + c] = h2f(tr[c]);
    return;
  }
  const uint16_t* pr = pos_table + (pos0 + r % rows_per_seq + pos_offset) * d;
  for (int64_t c = threadIdx.x; c < d; c += 256) x[r * d + c] = h2f(tr[c]) + h2f(pr[c]);
}

// Rotary positions.  Each thread turns 4 consecutive pairs (i, i + D/2) of
// one head of one row: (a, b) -> (a cos - b sin, b cos + a sin), in fp32 from
// fp16 and back (q also times q_scale before its one rounding).  Items of a
// row: the H query heads, then the Hkv key heads, D/8 items per head.
__global__ __launch_bounds__(256) void rope_k(uint16_t* __restrict__ q, uint16_t* __restrict__ k,
                                              const float* __restrict__ cs, int64_t M,
                                              int64_t rows_per_seq, int64_t pos0, int64_t kpos0,
                                              int64_t batch, int H, int Hkv, int D,
                                              float q_scale) {
  const int per_head = D / 8, per_row = (H + Hkv) * per_head;
  const int64_t item = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (item >= M * per_row) return;
  const int64_t m = item / per_row;
  const int r = (int)(item % per_row);
  const int hh = r / per_head, i = 4 * (r % per_head);
  const int64_t p = m % rows_per_seq, seq = m / rows_per_seq;
  uint16_t* base;
  float sc;
  if (hh < H) {
    base = q + m * ((int64_t)H * D) + (int64_t)hh * D;
    sc = q_scale;
  } else {
    base = k + ((kpos0 + p) * batch + seq) * ((int64_t)Hkv * D) + (int64_t)(hh - H) * D;
    sc = 1.f;
  }
  const float* c = cs + (pos0 + p) * D + 2 * i;  // D/2 (cos, sin) pairs per position
  const u32x2 av = *reinterpret_cast<const u32x2*>(base + i);
  const u32x2 bv = *reinterpret_cast<const u32x2*>(base + i + D / 2);
  u32x2 ao, bo;
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    uint32_t ra = 0, rb = 0;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int j = 2 * w + e;
      const float a = h2f((uint16_t)(av[w] >> (16 * e)));
      const float b = h2f((uint16_t)(bv[w] >> (16 * e)));
      const float co = c[2 * j], si = c[2 * j + 1];
      ra |= (uint32_t)f2h((a * co - b * si) * sc) << (16 * e);
      rb |= (uint32_t)f2h((b * co + a * si) * sc) << (16 * e);
    }
    ao[w] = ra;
    bo[w] = rb;
  }
  *reinterpret_cast<u32x2*>(base + i) = ao;
  *reinterpret_cast<u32x2*>(base + i + D / 2) = bo;
}

// SwiGLU: h[m][i] = silu(g) * u with g = gu[m][i], u = gu[m][F + i] and
// silu(g) = g / (1 + exp(-g)), in fp32; 8 elements per thread
__global__ __launch_bounds__(256) void swiglu_k(const uint16_t* __restrict__ gu,
                                                uint16_t* __restrict__ h, int64_t M, int64_t F) {
  const int64_t per_row = F / 8;
  const int64_t item = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (item >= M * per_row) return;
  const int64_t m = item / per_row, i = 8 * (item % per_row);
  const h8 g = load_h8(gu + m * 2 * F + i);
  const h8 u = load_h8(gu + m * 2 * F + F + i);
  u32x4 out;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t r = 0;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float gv = (float)g[2 * w + e], uv = (float)u[2 * w + e];
      r |= (uint32_t)f2h(gv / (1.f + expf(-gv)) * uv) << (16 * e);
    }
    out[w] = r;
  }
  *reinterpret_cast<u32x4*>(h + m * F + i) = out;
}

// greedy token: largest logit, ties to the lowest index (NaNs are skipped).
// A candidate (v, i) replaces (best, idx) if v > best, or v == best and
// i < idx; the result does not depend on the order candidates are seen.
__device__ __forceinline__ void argmax_take(float& best, int& idx, float v, int i) {
  if (v > best || (v == best && i < idx)) {
    best = v;
    idx = i;
  }
}

// best of a 256-thread block, written by thread 0
__device__ __forceinline__ void argmax_block(float& best, int& idx, float* bv, int* bi) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off, 64);
    const int oi = __shfl_xor(idx, off, 64);
    argmax_take(best, idx, ov, oi);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    bv[wave] = best;
    bi[wave] = idx;
  }
  __syncthreads();
  if (threadIdx.x == 0)
    for (int w = 1; w < 4; ++w) argmax_take(best, idx, bv[w], bi[w]);
}

// partition p of row `row` (grid (P, rows)): columns [p chunk, (p+1) chunk),
// four independent loads in flight per thread; the candidate goes to
// cand[row][p] (P == 1: straight to next[row])
__global__ __launch_bounds__(256) void argmax_k(const float* __restrict__ logits,
                                                int32_t* __restrict__ next,
                                                float2* __restrict__ cand, int64_t V,
                                                int64_t chunk) {
  __shared__ float bv[4];
  __shared__ int bi[4];
  const int64_t row = blockIdx.y, p = blockIdx.x, P = gridDim.x;
  const float* lr = logits + row * V;
  const int64_t lo = p * chunk, hi = min(V, lo + chunk);
  float best = -INFINITY;
  int idx = INT_MAX;
  for (int64_t i = lo + threadIdx.x; i < hi; i += 1024) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = i + 256 * u < hi ? lr[i + 256 * u] : NAN;
#pragma unroll
    for (int u = 0; u < 4; ++u) argmax_take(best, idx, v[u], (int)(i + 256 * u));
  }
  argmax_block(best, idx, bv, bi);
  if (threadIdx.x == 0) {
    if (P == 1)
      next[row] = idx == INT_MAX ? 0 : idx;
    else
      cand[row * P + p] = make_float2(best, __int_as_float(idx));
  }
}

// merge the P <= 64 candidates of each row (one wave per row)
__global__ __launch_bounds__(64) void argmax_merge_k(const float2* __restrict__ cand,
                                                     int32_t* __restrict__ next, int P) {
  const int64_t row = blockIdx.x;
  float best = -INFINITY;
  int idx = INT_MAX;
  if ((int)threadIdx.x < P) {
    const float2 c = cand[row * P + threadIdx.x];
    best = c.x;
    idx = __float_as_int(c.y);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off, 64);
    const int oi = __shfl_xor(idx, off, 64);
    argmax_take(best, idx, ov, oi);
  }
  if (threadIdx.x == 0) next[row] = idx == INT_MAX ? 0 : idx;
}

// plain streaming copy, 16 bytes per thread per iteration
__global__ __launch_bounds__(256) void copy16_k(const u32x4* __restrict__ src,
                                                u32x4* __restrict__ dst, int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    dst[i] = src[i];
}

__global__ void fill_u16_k(uint16_t* p, uint16_t value, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = value;
}

// ---------------------------------------------------------------------------
pipo_status launch_layernorm(const float* x, const uint16_t* g, const uint16_t* b, uint16_t* y,
                             int64_t rows, int64_t d, int64_t src_stride, int64_t src_offset,
                             float eps, hipStream_t st) {
  if (rows < 1 || d < 4 || d % 4 != 0 || d > 256 * 4 * kLnMaxVec) {
    set_error("layernorm: unsupported rows=%lld d=%lld", (long long)rows, (long long)d);
    return PIPO_ERR_UNSUPPORTED;
  }
  launch(norm_k<false>, dim3((unsigned)rows), dim3(256), 0, st, x, g, b, y, d, src_stride,
         src_offset, eps);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_rmsnorm(const float* x, const uint16_t* g, uint16_t* y, int64_t rows,
                           int64_t d, int64_t src_stride, int64_t src_offset, float eps,
                           hipStream_t st) {
  if (rows < 1 || d < 4 || d % 4 != 0 || d > 256 * 4 * kLnMaxVec) {
    set_error("rmsnorm: unsupported rows=%lld d=%lld", (long long)rows, (long long)d);
    return PIPO_ERR_UNSUPPORTED;
  }
  launch(norm_k<true>, dim3((unsigned)rows), dim3(256), 0, st, x, g, (const uint16_t*)nullptr, y,
         d, src_stride, src_offset, eps);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_rope(uint16_t* q, uint16_t* k, const float* cs, int64_t M,
                        int64_t rows_per_seq, int64_t pos0, int64_t kpos0, int64_t batch, int H,
                        int Hkv, int D, float q_scale, hipStream_t st) {
  if (M < 1) return PIPO_OK;
  if ((D != 64 && D != 128) || H < 1 || Hkv < 1 || rows_per_seq < 1 || batch < 1 || pos0 < 0 ||
      kpos0 < 0 || M > rows_per_seq * batch) {
    set_error("rope: unsupported shape M=%lld head_dim=%d heads=%d/%d", (long long)M, D, H, Hkv);
    return PIPO_ERR_UNSUPPORTED;
  }
  const int64_t items = M * (H + Hkv) * (D / 8);
  launch(rope_k, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, q, k, cs, M,
         rows_per_seq, pos0, kpos0, batch, H, Hkv, D, q_scale);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_swiglu(const uint16_t* gu, uint16_t* h, int64_t M, int64_t F, hipStream_t st) {
  if (M < 1) return PIPO_OK;
  if (F < 8 || F % 8 != 0) {
    set_error("swiglu: F=%lld is not a multiple of 8", (long long)F);
    return PIPO_ERR_UNSUPPORTED;
  }
  const int64_t items = M * (F / 8);
  launch(swiglu_k, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, gu, h, M, F);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_embed(const uint16_t* tok_rows, const int32_t* ids, const uint16_t* tok_table,
                         const uint16_t* pos_table, float* x, int64_t rows, int64_t d,
                         int64_t rows_per_seq, int64_t pos0, int64_t pos_offset, hipStream_t st) {
  if (rows < 1) return PIPO_OK;
  launch(embed_k, dim3((unsigned)rows), dim3(256), 0, st, tok_rows, ids, tok_table,
                     pos_table, x, d, rows_per_seq, pos0, pos_offset);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

// partitions of a row: about 4096 columns each, at most 64
static int argmax_parts(int64_t V) {
  const int64_t p = (V + 4095) / 4096;
  return (int)(p < 1 ? 1 : (p > 64 ? 64 : p));
}

int64_t argmax_workspace_bytes(int64_t rows, int64_t V) {
  const int P = argmax_parts(V);
  return P > 1 ? rows * P * (int64_t)sizeof(float2) : 0;
}

pipo_status launch_argmax(const float* logits, int32_t* next, int64_t rows, int64_t V,
                          void* workspace, int64_t workspace_bytes, hipStream_t st) {
  if (rows < 1 || V < 1 || V > INT_MAX || rows > 65535) {
    set_error("argmax: bad shape rows=%lld V=%lld", (long long)rows, (long long)V);
    return PIPO_ERR_ARG;
  }
  int P = argmax_parts(V);
  if (!workspace || workspace_bytes < argmax_workspace_bytes(rows, V)) P = 1;
  const int64_t chunk = (V + P - 1) / P;
  launch(argmax_k, dim3((unsigned)P, (unsigned)rows), dim3(256), 0, st, logits, next,
         static_cast<float2*>(workspace), V, chunk);
  if (P > 1)
    launch(argmax_merge_k, dim3((unsigned)rows), dim3(64), 0, st,
           static_cast<const float2*>(workspace), next, P);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_copy16(void* dst, const void* src, int64_t bytes, hipStream_t st) {
  if (bytes < 0 || bytes % 16 != 0 || ((uintptr_t)dst | (uintptr_t)src) % 16 != 0) {
    set_error("copy: %lld bytes or pointers not 16-byte aligned", (long long)bytes);
    return PIPO_ERR_ARG;
  }
  if (bytes == 0) return PIPO_OK;
  const int64_t n16 = bytes / 16;
  int64_t blocks = (n16 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  launch(copy16_k, dim3((unsigned)blocks), dim3(256), 0, st,
                     reinterpret_cast<const u32x4*>(src), reinterpret_cast<u32x4*>(dst), n16);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_fill_u16(uint16_t* p, uint16_t value, int64_t n, hipStream_t st) {
  if (n <= 0) return PIPO_OK;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  launch(fill_u16_k, dim3((unsigned)blocks), dim3(256), 0, st, p, value, n);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

}  // namespace pipo
