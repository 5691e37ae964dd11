// Causal softmax attention over a position-major KV cache: row p * b + i
// of K (or V) holds sequence i's key (value) at position p, all heads side
// by side.  This is the layout the copy engine streams when the cache lives
// in host memory: a layer's prefix 0..t-1 is one contiguous range.
//
//   attn_decode:  one new query per (sequence, head) against keys 0..t.
//   attn_prefill: P queries per (sequence, head), causal, flash-style with
//                 v_mfma_f32_16x16x32_f16 for Q K^T and P V.
// Softmax is max-subtracted in fp32; every reduction has a fixed order.
#include <algorithm>
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
// decode: grid (heads, b, splits), 256 threads.  Split z of a (sequence,
// head) covers keys [z * chunk, min(T, (z + 1) * chunk)).  A key is handled
// by D/8 lanes (8 dims each); every lane group keeps its own online softmax
// state (running max m, sum l, 8 accumulators) over the keys it visits, two
// keys at a time so that K and V of both are in flight together.  Groups are
// merged by a butterfly inside the wave, waves in order through LDS.  With
// one split the result is final; otherwise (m, l, acc[D]) goes to `part`
// and attn_decode_combine merges the splits in split order.  With KV4 the
// cache rows are INT4 (d/2 code bytes, then d/64 fp16 (scale, min) pairs):
// a lane reads its 8 codes and its group's pair and expands them to fp16.
template <int D>
__device__ __forceinline__ void online_merge(float& m, float& l, float (&acc)[8], float m2,
                                             float l2, const float (&acc2)[8]) {
  const float M = fmaxf(m, m2);
  const float a1 = m == -INFINITY ? 0.f : expf(m - M);
  const float a2 = m2 == -INFINITY ? 0.f : expf(m2 - M);
  l = l * a1 + l2 * a2;
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = acc[i] * a1 + acc2[i] * a2;
  m = M;
}

template <int D, bool KV4>
__global__ __launch_bounds__(256) void attn_decode_k(const uint16_t* __restrict__ q,
                                                     const void* __restrict__ kc,
                                                     const void* __restrict__ vc,
                                                     uint16_t* __restrict__ o,
                                                     float* __restrict__ part, int b, int H,
                                                     int t, int chunk) {
  __shared__ float wm[4], wl[4];
  __shared__ float wacc[4][D];
  constexpr int LPP = D / 8;     // lanes per key
  constexpr int PPW = 64 / LPP;  // keys per wave per pass
  const int h = blockIdx.x, bi = blockIdx.y, sp = blockIdx.z, S = gridDim.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane / LPP, cl = lane % LPP;
  const int64_t d = (int64_t)H * D;
  const int T = t + 1;
  const int p0 = sp * chunk, p1 = min(T, p0 + chunk);
  const int64_t col = (int64_t)h * D + cl * 8;

  float qf[8];
  {
    const h8 qv = load_h8(q + (int64_t)bi * d + col);
#pragma unroll
    for (int i = 0; i < 8; ++i) qf[i] = (float)qv[i];
  }
  float m = -INFINITY, l = 0.f, acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;

  // fp16: element offset of this lane's 8 values in row `bi` of position 0;
  // INT4: byte offsets of its 4 code bytes and of its group's (scale, min)
  const int64_t row_bytes = KV4 ? d / 2 + d / 16 : 2 * d;
  const int64_t code_off = (int64_t)bi * row_bytes + (KV4 ? col / 2 : 2 * col);
  const int64_t sm_off = (int64_t)bi * row_bytes + d / 2 + (col / 64) * 4;
  const auto load_kv = [&](const void* base, int p) -> h8 {
    const char* row = static_cast<const char*>(base) + (int64_t)p * b * row_bytes;
    if constexpr (KV4) {
      h2 s2, m2;
      scale_min_pairs(*reinterpret_cast<const uint32_t*>(row + sm_off), s2, m2);
      return dequant8(*reinterpret_cast<const uint32_t*>(row + code_off), s2, m2);
    } else {
      return load_h8(reinterpret_cast<const uint16_t*>(row + code_off));
    }
  };
  const auto visit = [&](h8 kv, h8 vv) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += qf[i] * (float)kv[i];
#pragma unroll
    for (int off = LPP / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    const float mn = fmaxf(m, s);
    const float alpha = expf(m - mn);
    const float e = expf(s - mn);
    l = l * alpha + e;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = acc[i] * alpha + e * (float)vv[i];
    m = mn;
  };
  for (int p = p0 + wave * PPW + sub; p < p1; p += 8 * PPW) {
    const int p2 = p + 4 * PPW;
    const h8 ka = load_kv(kc, p);
    const h8 va = load_kv(vc, p);
    h8 kb2 = zero_h8(), vb2 = zero_h8();
    if (p2 < p1) {
      kb2 = load_kv(kc, p2);
      vb2 = load_kv(vc, p2);
    }
    visit(ka, va);
    if (p2 < p1) visit(kb2, vb2);
  }
  // merge the lane groups of the wave (butterfly over the group index)
#pragma unroll
  for (int off = LPP; off < 64; off <<= 1) {
    float acc2[8];
    const float m2 = __shfl_xor(m, off, 64);
    const float l2 = __shfl_xor(l, off, 64);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc2[i] = __shfl_xor(acc[i], off, 64);
    online_merge<D>(m, l, acc, m2, l2, acc2);
  }
  if (sub == 0) {
    if (cl == 0) {
      wm[wave] = m;
      wl[wave] = l;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) wacc[wave][cl * 8 + i] = acc[i];
  }
  __syncthreads();
  for (int c = tid; c < D; c += 256) {
    float M = wm[0], L = wl[0], A = wacc[0][c];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float m2 = wm[w];
      const float Mn = fmaxf(M, m2);
      const float a1 = M == -INFINITY ? 0.f : expf(M - Mn);
      const float a2 = m2 == -INFINITY ? 0.f : expf(m2 - Mn);
      L = L * a1 + wl[w] * a2;
      A = A * a1 + wacc[w][c] * a2;
      M = Mn;
    }
    if (S == 1) {
      o[(int64_t)bi * d + (int64_t)h * D + c] = f2h(A / L);
    } else {
      float* pp = part + (((int64_t)bi * H + h) * S + sp) * (D + 2);
      pp[c] = A;
      if (c == 0) {
        pp[D] = M;
        pp[D + 1] = L;
      }
    }
  }
}

// merge the splits of each (sequence, head) in split order
template <int D>
__global__ __launch_bounds__(D) void attn_decode_combine(const float* __restrict__ part,
                                                         uint16_t* __restrict__ o, int H,
                                                         int S) {
  const int h = blockIdx.x, bi = blockIdx.y, c = threadIdx.x;
  const float* pp = part + ((int64_t)bi * H + h) * S * (D + 2);
  float M = pp[D], L = pp[D + 1], A = pp[c];
  for (int z = 1; z < S; ++z) {
    const float* pz = pp + (int64_t)z * (D + 2);
    const float m2 = pz[D];
    const float Mn = fmaxf(M, m2);
    const float a1 = M == -INFINITY ? 0.f : expf(M - Mn);
    const float a2 = m2 == -INFINITY ? 0.f : expf(m2 - Mn);
    L = L * a1 + pz[D + 1] * a2;
    A = A * a1 + pz[c] * a2;
    M = Mn;
  }
  o[((int64_t)bi * H + h) * D + c] = f2h(A / L);
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
int attn_decode_splits(int b, int n_heads, int t) {
  // enough workgroups to fill the chip, at least 64 keys per split
  const int T = t + 1;
  int S = (2048 + b * n_heads - 1) / (b * n_heads);
  S = std::min(S, std::max(1, T / 64));
  S = std::min(S, kAttnDecodeMaxSplits);
  const int chunk = (T + S - 1) / S;
  return (T + chunk - 1) / chunk;
}

int64_t attn_decode_workspace_bytes(int b, int n_heads, int head_dim, int splits) {
  return splits > 1 ? (int64_t)b * n_heads * splits * (head_dim + 2) * 4 : 0;
}

template <int D, bool KV4>
static void launch_decode_d(const uint16_t* q, const void* kc, const void* vc, uint16_t* o, int b,
                            int n_heads, int t, int S, int chunk, float* workspace,
                            hipStream_t st) {
  const dim3 grid((unsigned)n_heads, (unsigned)b, (unsigned)S);
  launch(attn_decode_k<D, KV4>, grid, dim3(256), 0, st, q, kc, vc, o, workspace, b, n_heads, t,
         chunk);
  if (S > 1)
    launch(attn_decode_combine<D>, dim3((unsigned)n_heads, (unsigned)b), dim3(D), 0, st,
           (const float*)workspace, o, n_heads, S);
}

pipo_status launch_attn_decode(const uint16_t* q, const void* kc, const void* vc, uint16_t* o,
                               int b, int n_heads, int head_dim, int t, bool kv4,
                               float* workspace, int64_t workspace_bytes, hipStream_t st) {
  if (b < 1 || n_heads < 1 || t < 0) {
    set_error("attn_decode: bad shape b=%d heads=%d t=%d", b, n_heads, t);
    return PIPO_ERR_ARG;
  }
  if (head_dim != 64 && head_dim != 128) {
    set_error("attn_decode: head_dim %d not supported (64 or 128)", head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (kv4 && ((int64_t)n_heads * head_dim) % 256 != 0) {
    set_error("attn_decode: INT4 KV rows need d %% 256 == 0 (d=%d)", n_heads * head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  const int T = t + 1;
  int S = attn_decode_splits(b, n_heads, t);
  if (!workspace || workspace_bytes < attn_decode_workspace_bytes(b, n_heads, head_dim, S)) S = 1;
  const int chunk = (T + S - 1) / S;
  S = (T + chunk - 1) / chunk;
  if (head_dim == 128)
    (kv4 ? launch_decode_d<128, true> : launch_decode_d<128, false>)(q, kc, vc, o, b, n_heads, t,
                                                                    S, chunk, workspace, st);
  else
    (kv4 ? launch_decode_d<64, true> : launch_decode_d<64, false>)(q, kc, vc, o, b, n_heads, t, S,
                                                                  chunk, workspace, st);
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
    launch(attn_prefill_k<128>, grid, dim3(256), 0, st, q, kc, vc, o, b, P, n_heads);
  } else if (head_dim == 64) {
    launch(attn_prefill_k<64>, grid, dim3(256), 0, st, q, kc, vc, o, b, P, n_heads);
  } else {
    set_error("attn_prefill: head_dim %d not supported (64 or 128)", head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

}  // namespace pipo
