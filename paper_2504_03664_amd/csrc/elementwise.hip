// Row-wise kernels of the decoder: LayerNorm, embedding, greedy argmax, and
// a fill used to poison weight slots.  The residual stream x is fp32; the
// LayerNorm output that feeds the next GEMM is fp16.
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

// y[r] = (x[src] - mean) / sqrt(var + eps) * gamma + beta, two passes over
// the row held in registers (d <= 256 * 4 * kLnMaxVec)
constexpr int kLnMaxVec = 8;

__global__ __launch_bounds__(256) void layernorm_k(const float* __restrict__ x,
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
  const float mean = block_sum256(s, red) / (float)d;
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
        const float a0 = (v[i][e] - mean) * rstd * h2f(gamma[k]) + h2f(beta[k]);
        const float a1 = (v[i][e + 1] - mean) * rstd * h2f(gamma[k + 1]) + h2f(beta[k + 1]);
        packed[e / 2] = (uint32_t)f2h(a0) | ((uint32_t)f2h(a1) << 16);
      }
      *reinterpret_cast<u32x2*>(yr + 4 * (int64_t)c) = packed;
    }
  }
}

// x[r][:] = tok(r) + pos_table[pos0 + r % rows_per_seq + pos_offset], with
// tok(r) = tok_rows[r] (gathered on the host) or tok_table[ids[r]]
__global__ __launch_bounds__(256) void embed_k(const uint16_t* __restrict__ tok_rows,
                                               const int32_t* __restrict__ ids,
                                               const uint16_t* __restrict__ tok_table,
                                               const uint16_t* __restrict__ pos_table,
                                               float* __restrict__ x, int64_t d,
                                               int64_t rows_per_seq, int64_t pos0,
                                               int64_t pos_offset) {
  const int64_t r = blockIdx.x;
  const uint16_t* tr = tok_rows ? tok_rows + r * d : tok_table + (int64_t)ids[r] * d;
  const uint16_t* pr = pos_table + (pos0 + r % rows_per_seq + pos_offset) * d;
  for (int64_t c = threadIdx.x; c < d; c += 256) x[r * d + c] = h2f(tr[c]) + h2f(pr[c]);
}

// greedy token: largest logit, ties to the lowest index (NaNs are skipped)
__global__ __launch_bounds__(256) void argmax_k(const float* __restrict__ logits,
                                                int32_t* __restrict__ next, int64_t V) {
  __shared__ float bv[4];
  __shared__ int bi[4];
  const int64_t row = blockIdx.x;
  const float* lr = logits + row * V;
  float best = -INFINITY;
  int idx = INT_MAX;
  for (int64_t i = threadIdx.x; i < V; i += 256) {
    const float v = lr[i];
    if (v > best || (idx == INT_MAX && v == best)) {
      best = v;
      idx = (int)i;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off, 64);
    const int oi = __shfl_xor(idx, off, 64);
    if (ov > best || (ov == best && oi < idx)) {
      best = ov;
      idx = oi;
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    bv[wave] = best;
    bi[wave] = idx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float b = bv[0];
    int k = bi[0];
    for (int w = 1; w < 4; ++w)
      if (bv[w] > b || (bv[w] == b && bi[w] < k)) {
        b = bv[w];
        k = bi[w];
      }
    next[row] = k == INT_MAX ? 0 : k;
  }
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
  launch(layernorm_k, dim3((unsigned)rows), dim3(256), 0, st, x, g, b, y, d,
                     src_stride, src_offset, eps);
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

pipo_status launch_argmax(const float* logits, int32_t* next, int64_t rows, int64_t V,
                          hipStream_t st) {
  if (rows < 1 || V < 1 || V > INT_MAX) {
    set_error("argmax: bad shape rows=%lld V=%lld", (long long)rows, (long long)V);
    return PIPO_ERR_ARG;
  }
  launch(argmax_k, dim3((unsigned)rows), dim3(256), 0, st, logits, next, V);
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
