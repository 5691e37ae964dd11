// Causal softmax attention over a position-major KV cache: row p * b + i
// of K (or V) holds sequence i's key (value) at position p, all key/value
// heads side by side.  With grouped-query attention, query head h reads
// key/value head h / (H / Hkv).  This is the layout the copy engine streams when the cache lives
// in host memory: a layer's prefix 0..t-1 is one contiguous range.
//
//   attn_decode:  one new query per (sequence, head) against keys 0..t.
//   attn_prefill: P queries per (sequence, head), causal, flash-style with
//                 v_mfma_f32_16x16x32_f16 for Q K^T and P V.
// Softmax is max-subtracted in fp32; every reduction has a fixed order.
#include <algorithm>
#include <cfloat>
#include <mutex>

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

// Sum over aligned groups of N <= 16 lanes with DPP moves inside a row of 16
// lanes (swap neighbours, swap pairs, mirror within 8, mirror within 16):
// ALU operations instead of the LDS round trips of lane shuffles.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __uint_as_float(
      __builtin_amdgcn_update_dpp(0u, __float_as_uint(v), CTRL, 0xF, 0xF, false));
}
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16, "groups of up to 16 lanes");
  if constexpr (N >= 2) v += dpp_move<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  if constexpr (N >= 4) v += dpp_move<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  if constexpr (N >= 8) v += dpp_move<0x141>(v);  // row_half_mirror
  if constexpr (N >= 16) v += dpp_move<0x140>(v); // row_mirror
  return v;
}

// ---------------------------------------------------------------------------
// decode: grid (key/value head groups, b, splits), 256 threads.  A workgroup
// serves HP adjacent key/value heads of one sequence and the G = H / Hkv
// query heads that read each of them (HP > 1 only without grouping, G = 1),
// so each cached row is read from HBM once per step and a key's HP heads
// are one contiguous HP * D * 2-byte read.  Split z of a (sequence, head
// group) covers keys [z * chunk, min(T, (z + 1) * chunk)).  A key's head is
// handled by D/8 lanes (8 dims each; fp16 rows are read with non-temporal
// loads, as every row is read once); every lane group keeps, per query
// head, its own online softmax state (running max m, sum l, 8 accumulators)
// over the keys it visits, two keys at a time so that K and V of both are
// in flight together (the second one's index is clamped, so the loads are
// unconditional).  Groups are merged by a butterfly inside the wave, waves
// in order through LDS.  With one split the result is final; otherwise (m,
// l, acc[D]) of each query head goes to `part` and attn_decode_combine
// merges the splits in split order.  With KV4 the cache rows are INT4
// (dkv/2 code bytes, then dkv/64 fp16 (scale, min) pairs): a lane reads its
// 8 codes and its group's pair and expands them to fp16.
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

template <int D, int G, int HP, bool KV4>
__global__ __launch_bounds__(256) void attn_decode_k(const uint16_t* __restrict__ q,
                                                     const void* __restrict__ kc,
                                                     const void* __restrict__ vc,
                                                     uint16_t* __restrict__ o,
                                                     float* __restrict__ part, int b, int Hkv,
                                                     int t, int chunk) {
  static_assert(G == 1 || HP == 1, "several heads per workgroup only without grouping");
  constexpr float kLog2e = 1.4426950408889634f;
  constexpr int LPP = D / 8;      // lanes per head of a key
  constexpr int LPK = HP * LPP;   // lanes per key
  constexpr int PPW = 64 / LPK;   // keys per wave per pass
  constexpr int NQ = HP * G;      // query heads of the workgroup
  __shared__ float wm[4][NQ], wl[4][NQ];
  __shared__ float wacc[4][NQ * D];
  const int kb = blockIdx.x, bi = blockIdx.y, sp = blockIdx.z, S = gridDim.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane / LPK, cl = lane % LPK, hl = cl / LPP, cd = (cl % LPP) * 8;
  const int H = Hkv * G;
  const int64_t d = (int64_t)H * D, dkv = (int64_t)Hkv * D;
  const int T = t + 1;
  const int p0 = sp * chunk, p1 = min(T, p0 + chunk);
  const int kh = kb * HP + hl;                    // this lane's key/value head
  const int64_t kcol = (int64_t)kh * D + cd;

  float qf[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const h8 qv = load_h8(q + (int64_t)bi * d + (int64_t)(kh * G + g) * D + cd);
#pragma unroll
    for (int i = 0; i < 8; ++i) qf[g][i] = (float)qv[i];
  }
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[g][i] = 0.f;
  }

  // fp16: byte offset of this lane's 8 values in row `bi` of position 0;
  // INT4: byte offsets of its 4 code bytes and of its group's (scale, min)
  const int64_t row_bytes = KV4 ? dkv / 2 + dkv / 16 : 2 * dkv;
  const int64_t code_off = (int64_t)bi * row_bytes + (KV4 ? kcol / 2 : 2 * kcol);
  const int64_t sm_off = (int64_t)bi * row_bytes + dkv / 2 + (kcol / 64) * 4;
  const auto load_kv = [&](const void* base, int p) -> h8 {
    const char* row = static_cast<const char*>(base) + (int64_t)p * b * row_bytes;
    if constexpr (KV4) {
      h2 s2, m2;
      scale_min_pairs(*reinterpret_cast<const uint32_t*>(row + sm_off), s2, m2);
      return dequant8(*reinterpret_cast<const uint32_t*>(row + code_off), s2, m2);
    } else {
      return load_h8_stream(reinterpret_cast<const uint16_t*>(row + code_off));
    }
  };
  const auto visit = [&](h8 kv, h8 vv) {
    float kf[8], vf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      kf[i] = (float)kv[i];
      vf[i] = (float)vv[i];
    }
    if constexpr (G == 1) {  // bound by HBM: the plain update (DPP sums measured no faster)
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) s += qf[0][i] * kf[i];
#pragma unroll
      for (int off = LPP / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
      const float mn = fmaxf(m[0], s);
      const float alpha = expf(m[0] - mn);
      const float e = expf(s - mn);
      l[0] = l[0] * alpha + e;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[0][i] = acc[0][i] * alpha + e * vf[i];
      m[0] = mn;
    } else {  // G query heads per key: bound by arithmetic
      float alpha[G], e[G];
      bool grew = false;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += qf[g][i] * kf[i];
        s = group_sum<LPP>(s);
        const float mn = fmaxf(m[g], s);
        // hardware exp2; m = -inf on the first key gives alpha = 0
        alpha[g] = __builtin_amdgcn_exp2f((m[g] - mn) * kLog2e);
        e[g] = __builtin_amdgcn_exp2f((s - mn) * kLog2e);
        l[g] = l[g] * alpha[g] + e[g];
        grew |= alpha[g] != 1.f;
        m[g] = mn;
      }
      // the running maxima rarely grow after the first keys: rescale only
      // when some lane's did (alpha = 1 exactly otherwise)
      if (__any(grew)) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[g][i] *= alpha[g];
      }
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[g][i] += e[g] * vf[i];
    }
  };
  for (int p = p0 + wave * PPW + sub; p < p1; p += 8 * PPW) {
    const int p2 = min(p + 4 * PPW, p1 - 1);
    const h8 ka = load_kv(kc, p);
    const h8 va = load_kv(vc, p);
    const h8 kb2 = load_kv(kc, p2);
    const h8 vb2 = load_kv(vc, p2);
    visit(ka, va);
    if (p + 4 * PPW < p1) visit(kb2, vb2);
  }
  // merge the lane groups of the wave (butterfly over the group index)
#pragma unroll
  for (int off = LPK; off < 64; off <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float acc2[8];
      const float m2 = __shfl_xor(m[g], off, 64);
      const float l2 = __shfl_xor(l[g], off, 64);
#pragma unroll
      for (int i = 0; i < 8; ++i) acc2[i] = __shfl_xor(acc[g][i], off, 64);
      online_merge(m[g], l[g], acc[g], m2, l2, acc2);
    }
  }
  if (sub == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int j = hl * G + g;  // query head within the workgroup
      if (cd == 0) {
        wm[wave][j] = m[g];
        wl[wave][j] = l[g];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) wacc[wave][j * D + cd + i] = acc[g][i];
    }
  }
  __syncthreads();
  for (int c = tid; c < NQ * D; c += 256) {
    const int j = c / D, cc = c % D, h = kb * NQ + j;
    float M = wm[0][j], L = wl[0][j], A = wacc[0][c];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float m2 = wm[w][j];
      const float Mn = fmaxf(M, m2);
      const float a1 = M == -INFINITY ? 0.f : expf(M - Mn);
      const float a2 = m2 == -INFINITY ? 0.f : expf(m2 - Mn);
      L = L * a1 + wl[w][j] * a2;
      A = A * a1 + wacc[w][c] * a2;
      M = Mn;
    }
    if (S == 1) {
      o[(int64_t)bi * d + (int64_t)h * D + cc] = f2h(A / L);
    } else {
      float* pp = part + (((int64_t)bi * H + h) * S + sp) * (D + 2);
      pp[cc] = A;
      if (cc == 0) {
        pp[D] = M;
        pp[D + 1] = L;
      }
    }
  }
}

// decode over an INT4 cache without grouping (G = 1): the same structure
// as attn_decode_k, but a lane holds 32 elements of a key's head (one
// 16-byte load of codes and one (scale, min) pair instead of four 4-byte
// loads for 8 elements each), so a wave issues a quarter of the load
// instructions per byte; D/32 lanes per head of a key.  The kernel is
// bound by its arithmetic, so codes are expanded in pairs (k, k + 4) of
// each group of 8 (one shift and mask per pair), q is held as fp16 pairs
// in that order for two-element dot products (v_dot2_f32_f16), the
// accumulators follow the same order until they are stored, and the
// softmax uses the hardware exp2.
template <int D, int HP>
__global__ __launch_bounds__(256) void attn_decode_kv4_k(const uint16_t* __restrict__ q,
                                                         const void* __restrict__ kc,
                                                         const void* __restrict__ vc,
                                                         uint16_t* __restrict__ o,
                                                         float* __restrict__ part, int b, int H,
                                                         int t, int chunk) {
  constexpr int EPL = 32;            // elements per lane
  constexpr int LPP = D / EPL;       // lanes per head of a key
  constexpr int LPK = HP * LPP;      // lanes per key
  constexpr int PPW = 64 / LPK;      // keys per wave per pass
  __shared__ float wm[4][HP], wl[4][HP];
  __shared__ float wacc[4][HP * D];
  const int kb = blockIdx.x, bi = blockIdx.y, sp = blockIdx.z, S = gridDim.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane / LPK, cl = lane % LPK, hl = cl / LPP, cd = (cl % LPP) * EPL;
  const int64_t d = (int64_t)H * D;
  const int T = t + 1;
  const int p0 = sp * chunk, p1 = min(T, p0 + chunk);
  const int64_t col = (int64_t)(kb * HP + hl) * D + cd;

  constexpr float kLog2e = 1.4426950408889634f;
  // qh[4 j + u] = (q[8 j + u], q[8 j + u + 4]); acc[8 j + 2 u + h] is element
  // 8 j + u + 4 h
  h2 qh[EPL / 2];
#pragma unroll
  for (int j = 0; j < EPL / 8; ++j) {
    const h8 qi = interleave_h8(load_h8(q + (int64_t)bi * d + col + 8 * j));
#pragma unroll
    for (int u = 0; u < 4; ++u) qh[4 * j + u] = h2{qi[2 * u], qi[2 * u + 1]};
  }
  float m = -INFINITY, l = 0.f, acc[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) acc[i] = 0.f;

  const int64_t row_bytes = d / 2 + d / 16;
  const int64_t code_off = (int64_t)bi * row_bytes + col / 2;            // 16-byte aligned
  const int64_t sm_off = (int64_t)bi * row_bytes + d / 2 + (col / 64) * 4;
  struct Row {
    u32x4 codes;
    uint32_t sm;
  };
  const auto load_row = [&](const void* base, int p) -> Row {
    const char* row = static_cast<const char*>(base) + (int64_t)p * b * row_bytes;
    return Row{*reinterpret_cast<const u32x4*>(row + code_off),
               *reinterpret_cast<const uint32_t*>(row + sm_off)};
  };
  const auto visit = [&](const Row& kr, const Row& vr) {
    h2 ks, km, vs, vm;
    scale_min_pairs(kr.sm, ks, km);
    scale_min_pairs(vr.sm, vs, vm);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        s = __builtin_amdgcn_fdot2(
            qh[4 * j + u], dequant_pair((kr.codes[j] >> (4 * u)) & 0x000F000Fu, ks, km), s, false);
    s = group_sum<LPP>(s);
    const float mn = fmaxf(m, s);
    // m = -inf on the first key: exp2(-inf) = 0
    const float alpha = __builtin_amdgcn_exp2f((m - mn) * kLog2e);
    const float e = __builtin_amdgcn_exp2f((s - mn) * kLog2e);
    l = l * alpha + e;
    // the running maxima rarely grow after the first keys: rescale only
    // when some lane's did (alpha = 1 exactly otherwise)
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int i = 0; i < EPL; ++i) acc[i] *= alpha;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const h2 vp = dequant_pair((vr.codes[j] >> (4 * u)) & 0x000F000Fu, vs, vm);
        acc[8 * j + 2 * u] += e * (float)vp[0];
        acc[8 * j + 2 * u + 1] += e * (float)vp[1];
      }
    m = mn;
  };
  for (int p = p0 + wave * PPW + sub; p < p1; p += 8 * PPW) {
    const int p2 = min(p + 4 * PPW, p1 - 1);
    const Row ka = load_row(kc, p), va = load_row(vc, p);
    const Row kb2 = load_row(kc, p2), vb2 = load_row(vc, p2);
    visit(ka, va);
    if (p + 4 * PPW < p1) visit(kb2, vb2);
  }
  // merge the key slots of the wave, then the waves through LDS
#pragma unroll
  for (int off = LPK; off < 64; off <<= 1) {
    const float m2 = __shfl_xor(m, off, 64);
    const float l2 = __shfl_xor(l, off, 64);
    const float M = fmaxf(m, m2);
    const float a1 = m == -INFINITY ? 0.f : expf(m - M);
    const float a2 = m2 == -INFINITY ? 0.f : expf(m2 - M);
    l = l * a1 + l2 * a2;
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] = acc[i] * a1 + __shfl_xor(acc[i], off, 64) * a2;
    m = M;
  }
  if (sub == 0) {
    if (cd == 0) {
      wm[wave][hl] = m;
      wl[wave][hl] = l;
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      wacc[wave][hl * D + cd + 8 * (i / 8) + (i % 8) / 2 + 4 * (i % 2)] = acc[i];
  }
  __syncthreads();
  for (int c = tid; c < HP * D; c += 256) {
    const int j = c / D, cc = c % D, h = kb * HP + j;
    float M = wm[0][j], L = wl[0][j], A = wacc[0][c];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float m2 = wm[w][j];
      const float Mn = fmaxf(M, m2);
      const float a1 = M == -INFINITY ? 0.f : expf(M - Mn);
      const float a2 = m2 == -INFINITY ? 0.f : expf(m2 - Mn);
      L = L * a1 + wl[w][j] * a2;
      A = A * a1 + wacc[w][c] * a2;
      M = Mn;
    }
    if (S == 1) {
      o[(int64_t)bi * d + (int64_t)h * D + cc] = f2h(A / L);
    } else {
      float* pp = part + (((int64_t)bi * H + h) * S + sp) * (D + 2);
      pp[cc] = A;
      if (cc == 0) {
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
// prefill (flash-style): a workgroup owns 128 queries of one head and
// sequence, 4 waves x 32 queries (two sub-blocks of 16).  Keys come in
// blocks of 64, K and V moved from the cache straight into LDS by the load
// unit (double-buffered), rows stored with their 16-byte chunks permuted by
// row (kv_swz) so that the K fragment reads and the transposed V reads hit
// distinct banks.  The wave
// computes S^T = K Q^T (keys on the MFMA rows, its queries on the columns,
// so each lane holds scores of one query), an online softmax per query in
// fp32, and O^T += V^T P^T: the probabilities stay in the registers they
// were computed in (a lane's 8 keys per MFMA are the ones its S^T fragment
// gave it; V^T is read with the same key order through transposed LDS
// reads).  Workgroups with the most key blocks start first.
constexpr int kPQ = 128;  // queries per workgroup
constexpr int kPK = 64;   // keys per block
constexpr int kPrefillStages = 2;

// LDS slot of 16-byte chunk `chunk` of key row `key` (an involution: the
// DMA puts cache chunk kv_swz(row, s) into slot s, a read of chunk c goes
// to slot kv_swz(row, c)).  The chunk is XORed with a mask that depends on
// the row's low four bits, chosen with the LDS bank-conflict counters: over
// the K fragment reads (ds_read_b128; lane r + 16 g reads row r of a 16-row
// group, chunk 4 kk + g) and the transposed V reads (ds_read_b64_tr_b16;
// rows 4 g .. 4 g + 3 of a group, chunks 2 n and 2 n + 1), a plain XOR with
// the row leaves the K reads conflict-free but gives every V read a 2-way
// conflict, the row rotated left by one bit the reverse, and of 240 random
// masks that clear the V reads three cleared the K reads as well; the table
// below is the first of them (head_dim 128: 16 chunks per row).  For
// head_dim 64 (two rows per 256 bytes) the mask row & 6 measured no
// conflicts on either read.
template <int D>
__device__ __forceinline__ int kv_swz(int key, int chunk) {
  if constexpr (D == 128) {
    constexpr uint64_t kMask = 0x618d34ea5b2f0c97ull;  // nibble x: mask of rows with key % 16 == x
    return chunk ^ (int)((kMask >> (4 * (key & 15))) & 15);
  } else {
    return chunk ^ (key & 6);
  }
}

// the pair of values that v_permlane16/32_swap leave in a lane: its own
// and that of the lane 16 (32) apart, in either order
template <typename P>
__device__ __forceinline__ float pair_max(P p) {
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
template <typename P>
__device__ __forceinline__ float pair_sum(P p) {
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

template <int NS, int DMA>
__device__ __forceinline__ void wait_blocks_landed(int pending) {
  // at most `pending` later blocks (2 DMA loads per wave each) outstanding
  if constexpr (NS >= 4) {
    if (pending >= 3) {
      __builtin_amdgcn_s_waitcnt(waitcnt_imm(3 * 2 * DMA, false));
      return;
    }
  }
  if constexpr (NS >= 3) {
    if (pending >= 2) {
      __builtin_amdgcn_s_waitcnt(waitcnt_imm(2 * 2 * DMA, false));
      return;
    }
  }
  if (pending >= 1) {
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(2 * DMA, false));
    return;
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, false));
}

template <int D, int NS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void attn_prefill_k(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ vc, uint16_t* __restrict__ o, int b, int P, int H, int Hkv) {
  constexpr int ROWB = 2 * D;               // bytes per key row in LDS
  constexpr int BLK = kPK * ROWB;           // bytes of K (or V) per block
  constexpr int DMA = BLK / 1024 / 4;       // DMA instructions per wave for K (and for V)
  constexpr int KK = D / 32;                // MFMA k steps over the head dimension
  constexpr int NF = D / 16;                // head-dimension fragments of O^T
  constexpr float kLog2e = 1.4426950408889634f;
  __shared__ __attribute__((aligned(1024))) uint8_t kv[NS][2][BLK];  // [stage][K, V]

  const int nqb = (P + kPQ - 1) / kPQ;
  const int qb = nqb - 1 - (int)blockIdx.x;  // most key blocks first
  const int h = blockIdx.y, bi = blockIdx.z;
  const int64_t d = (int64_t)H * D, dkv = (int64_t)Hkv * D;
  const int kh = h / (H / Hkv);
  // the wave index in a scalar register, so that everything derived from
  // it (the wave's queries, which blocks it masks) is wave-uniform
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, g = lane >> 4;
  const int qw = qb * kPQ + wave * 32;       // this wave's first query
  const int nkb = (min(qb * kPQ + kPQ, P) + kPK - 1) / kPK;

  // Q^T fragments (B operand): lane (r, g) holds query qw + 16 u + r, dims 32 kk + 8 g ..
  h8 qf[2][KK];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int qp = qw + 16 * u + r;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qf[u][kk] = qp < P ? load_h8(q + ((int64_t)bi * P + qp) * d + (int64_t)h * D + 32 * kk + 8 * g)
                         : zero_h8();
  }

  // DMA of key block kb into buffer buf: LDS byte p of a block holds row
  // p / ROWB, chunk slot (p % ROWB) / 16, i.e. cache chunk kv_swz(row, slot).
  // The block's first row is a wave-uniform address and a lane's offsets
  // from it do not depend on the block (32-bit: the host checks that a
  // block of rows spans less than 2^31 elements), so they are computed
  // once; only a block that reaches past P clamps its rows.
  const int row_elems = b * (int)dkv;  // elements between positions
  const uint16_t* kbase = kc + (int64_t)bi * dkv + (int64_t)kh * D;
  const uint16_t* vbase = vc + (int64_t)bi * dkv + (int64_t)kh * D;
  int doff[DMA];
#pragma unroll
  for (int i = 0; i < DMA; ++i) {
    const int p = (wave * DMA + i) * 1024 + lane * 16;
    doff[i] = (p / ROWB) * row_elems + 8 * kv_swz<D>(p / ROWB, (p % ROWB) / 16);
  }
  const auto issue = [&](int kb, int buf) {
    const int k0 = kb * kPK;
    const uint16_t* kblk = kbase + (int64_t)k0 * row_elems;
    const uint16_t* vblk = vbase + (int64_t)k0 * row_elems;
    const bool clamp = k0 + kPK > P;
#pragma unroll
    for (int i = 0; i < DMA; ++i) {
      int off = doff[i];
      if (clamp) {
        const int p = (wave * DMA + i) * 1024 + lane * 16, row = p / ROWB;
        off += (min(k0 + row, P - 1) - (k0 + row)) * row_elems;
      }
      lds_dma16(kblk + off, &kv[buf][0][(wave * DMA + i) * 1024]);
      lds_dma16(vblk + off, &kv[buf][1][(wave * DMA + i) * 1024]);
    }
  };

  f4 oacc[2][NF];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int n = 0; n < NF; ++n) oacc[u][n] = f4{0.f, 0.f, 0.f, 0.f};
  float mrow[2] = {-INFINITY, -INFINITY}, lrow[2] = {0.f, 0.f};

#pragma unroll
  for (int i = 0; i < NS; ++i)
    if (i < nkb) issue(i, i);
  for (int kb = 0; kb < nkb; ++kb) {
    const int buf = kb % NS;
    // block kb landed (blocks kb + 1 .. kb + NS - 1 may still be in flight)
    wait_blocks_landed<NS, DMA>(min(NS - 1, nkb - 1 - kb));
    wg_barrier();
    const int k0 = kb * kPK;
    if (k0 <= qw + 31) {  // some key of the block is visible to this wave
      const uint8_t* Kl = kv[buf][0];
      const uint8_t* Vl = kv[buf][1];
      // S^T: s[u][j][e] = score of key k0 + 16 j + 4 g + e for query qw + 16 u + r
      f4 s[2][4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        s[0][j] = f4{0.f, 0.f, 0.f, 0.f};
        s[1][j] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          const int row = 16 * j + r;
          const h8 kf = *reinterpret_cast<const h8*>(Kl + row * ROWB + 16 * kv_swz<D>(row, 4 * kk + g));
          s[0][j] = mfma16(kf, qf[0][kk], s[0][j]);
          s[1][j] = mfma16(kf, qf[1][kk], s[1][j]);
        }
      }
      // the block needs masking (a wave-uniform test)
      const bool edge = k0 + kPK - 1 > qw || k0 + kPK > P;
      if (edge) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int qp = qw + 16 * u + r;
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int key = k0 + 16 * j + 4 * g + e;
              s[u][j][e] = key > qp || key >= P ? -INFINITY : s[u][j][e];
            }
        }
      }
      h8 pf[2][2];  // P^T fragments (B operand) per sub-block and 32-key half
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float bm = -INFINITY;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) bm = fmaxf(bm, s[u][j][e]);
        bm = pair_max(__builtin_amdgcn_permlane16_swap(__float_as_uint(bm), __float_as_uint(bm), false, false));
        bm = pair_max(__builtin_amdgcn_permlane32_swap(__float_as_uint(bm), __float_as_uint(bm), false, false));
        const float mnew = fmaxf(mrow[u], bm);
        // every query row has a visible key in its first block, so mnew is finite
        const float alpha = exp2f((mrow[u] - mnew) * kLog2e);
        const float mb = mnew * kLog2e;
        mrow[u] = mnew;
        float rs = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            // v_exp_f32 without denormal scaling: p below 2^-126 becomes 0
            const float p = __builtin_amdgcn_exp2f(s[u][j][e] * kLog2e - mb);
            s[u][j][e] = p;
            rs += p;
          }
        rs = pair_sum(__builtin_amdgcn_permlane16_swap(__float_as_uint(rs), __float_as_uint(rs), false, false));
        rs = pair_sum(__builtin_amdgcn_permlane32_swap(__float_as_uint(rs), __float_as_uint(rs), false, false));
        lrow[u] = lrow[u] * alpha + rs;
        // after the first blocks the running maxima rarely grow: rescale
        // only when some lane's did (alpha is exactly 1 otherwise)
        if (__any(alpha != 1.f)) {
#pragma unroll
          for (int n = 0; n < NF; ++n) oacc[u][n] *= alpha;
        }
#pragma unroll
        for (int hk = 0; hk < 2; ++hk)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            pf[u][hk][e] = (_Float16)s[u][2 * hk][e];
            pf[u][hk][4 + e] = (_Float16)s[u][2 * hk + 1][e];
          }
      }
      // O^T += V^T P^T over the two 32-key halves: lane (r, g) needs V rows
      // 32 hk + 4 g + (0..3) and 32 hk + 16 + 4 g + (0..3), dim 16 n + r;
      // lane i' of its group addresses row base + i' / 4, dims 16 n + 4 (i' % 4)
#pragma unroll
      for (int hk = 0; hk < 2; ++hk)
#pragma unroll
        for (int n = 0; n < NF; ++n) {
          h8 vf;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const int row = 32 * hk + 16 * half + 4 * g + (r >> 2);
            const int dim = 16 * n + 4 * (r & 3);
            const h4 t = lds_read_tr16(Vl + row * ROWB + 16 * kv_swz<D>(row, dim / 8) + 2 * (dim % 8));
#pragma unroll
            for (int e = 0; e < 4; ++e) vf[4 * half + e] = t[e];
          }
          oacc[0][n] = mfma16(vf, pf[0][hk], oacc[0][n]);
          oacc[1][n] = mfma16(vf, pf[1][hk], oacc[1][n]);
        }
    }
    // every wave is done with this buffer
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, true));
    wg_barrier();
    if (kb + NS < nkb) issue(kb + NS, buf);
  }

  // oacc[u][n][e]: dim 16 n + 4 g + e of query qw + 16 u + r
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int qp = qw + 16 * u + r;
    if (qp >= P) continue;
    const float inv = 1.f / lrow[u];
    uint16_t* orow = o + ((int64_t)bi * P + qp) * d + (int64_t)h * D;
#pragma unroll
    for (int n = 0; n < NF; ++n) {
      u32x2 w;
      w[0] = (uint32_t)f2h(oacc[u][n][0] * inv) | ((uint32_t)f2h(oacc[u][n][1] * inv) << 16);
      w[1] = (uint32_t)f2h(oacc[u][n][2] * inv) | ((uint32_t)f2h(oacc[u][n][3] * inv) << 16);
      *reinterpret_cast<u32x2*>(orow + 16 * n + 4 * g) = w;
    }
  }
}

// ---------------------------------------------------------------------------
int attn_decode_heads_per_wg(int b, int n_heads, int n_kv_heads, bool kv4) {
  if (n_heads != n_kv_heads) return 1;
  int hp = n_heads % 4 == 0 ? 4 : (n_heads % 2 == 0 ? 2 : 1);
  // fp16 rows are bound by HBM: fewer heads per workgroup while that leaves
  // fewer than kAttnDecodeWideWGs workgroups (six per CU keep more loads in
  // flight than a longer key loop per wave).  INT4 rows are bound by the
  // expansion arithmetic, which the wide rows amortise better.
  if (!kv4)
    while (hp > 1 && (int64_t)b * (n_heads / hp) < kAttnDecodeWideWGs) hp /= 2;
  return hp;
}

int attn_decode_splits(int b, int n_heads, int n_kv_heads, int t, bool kv4) {
  // at least kAttnDecodeMinWGs workgroups (three per CU: fewer leave HBM
  // idle, more only add merge traffic), at least 64 keys per split
  const int T = t + 1;
  const int wgs = b * (n_kv_heads / attn_decode_heads_per_wg(b, n_heads, n_kv_heads, kv4));
  int S = (kAttnDecodeMinWGs + wgs - 1) / wgs;
  S = std::min(S, std::max(1, T / 64));
  S = std::min(S, kAttnDecodeMaxSplits);
  const int chunk = (T + S - 1) / S;
  return (T + chunk - 1) / chunk;
}

int64_t attn_decode_workspace_bytes(int b, int n_heads, int head_dim, int splits) {
  return splits > 1 ? (int64_t)b * n_heads * splits * (head_dim + 2) * 4 : 0;
}

template <int D, int G, int HP, bool KV4>
static void launch_decode_g(const uint16_t* q, const void* kc, const void* vc, uint16_t* o,
                            int b, int Hkv, int t, int S, int chunk, float* workspace,
                            hipStream_t st) {
  const dim3 grid((unsigned)(Hkv / HP), (unsigned)b, (unsigned)S);
  launch(attn_decode_k<D, G, HP, KV4>, grid, dim3(256), 0, st, q, kc, vc, o, workspace, b, Hkv,
         t, chunk);
  if (S > 1)
    launch(attn_decode_combine<D>, dim3((unsigned)(Hkv * G), (unsigned)b), dim3(D), 0, st,
           (const float*)workspace, o, Hkv * G, S);
}

template <int D, int HP>
static void launch_decode_kv4(const uint16_t* q, const void* kc, const void* vc, uint16_t* o,
                              int b, int H, int t, int S, int chunk, float* workspace,
                              hipStream_t st) {
  const dim3 grid((unsigned)(H / HP), (unsigned)b, (unsigned)S);
  launch(attn_decode_kv4_k<D, HP>, grid, dim3(256), 0, st, q, kc, vc, o, workspace, b, H, t,
         chunk);
  if (S > 1)
    launch(attn_decode_combine<D>, dim3((unsigned)H, (unsigned)b), dim3(D), 0, st,
           (const float*)workspace, o, H, S);
}

template <int D, bool KV4>
static void launch_decode_d(const uint16_t* q, const void* kc, const void* vc, uint16_t* o, int b,
                            int Hkv, int G, int HP, int t, int S, int chunk, float* workspace,
                            hipStream_t st) {
  if constexpr (KV4) {  // INT4 rows without grouping: 32 elements per lane
    if (G == 1) {
      if (HP == 4) return launch_decode_kv4<D, 4>(q, kc, vc, o, b, Hkv, t, S, chunk, workspace, st);
      if (HP == 2) return launch_decode_kv4<D, 2>(q, kc, vc, o, b, Hkv, t, S, chunk, workspace, st);
      return launch_decode_kv4<D, 1>(q, kc, vc, o, b, Hkv, t, S, chunk, workspace, st);
    }
  }
#define PIPO_DECODE_CASE(g, hp)                                                         \
  if (G == g && HP == hp)                                                               \
    return launch_decode_g<D, g, hp, KV4>(q, kc, vc, o, b, Hkv, t, S, chunk, workspace, \
                                          st);
  PIPO_DECODE_CASE(1, 4)
  PIPO_DECODE_CASE(1, 2)
  PIPO_DECODE_CASE(1, 1)
  PIPO_DECODE_CASE(2, 1)
  PIPO_DECODE_CASE(4, 1)
  PIPO_DECODE_CASE(8, 1)
#undef PIPO_DECODE_CASE
}

static pipo_status check_heads(const char* what, int n_heads, int n_kv_heads, int head_dim) {
  if (head_dim != 64 && head_dim != 128) {
    set_error("%s: head_dim %d not supported (64 or 128)", what, head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (n_kv_heads < 1 || n_heads % n_kv_heads != 0) {
    set_error("%s: %d query heads are not a multiple of %d key/value heads", what, n_heads,
              n_kv_heads);
    return PIPO_ERR_ARG;
  }
  const int G = n_heads / n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) {
    set_error("%s: %d query heads per key/value head not supported (1, 2, 4, 8)", what, G);
    return PIPO_ERR_UNSUPPORTED;
  }
  return PIPO_OK;
}

pipo_status launch_attn_decode(const uint16_t* q, const void* kc, const void* vc, uint16_t* o,
                               int b, int n_heads, int n_kv_heads, int head_dim, int t, bool kv4,
                               float* workspace, int64_t workspace_bytes, hipStream_t st) {
  if (b < 1 || n_heads < 1 || t < 0) {
    set_error("attn_decode: bad shape b=%d heads=%d t=%d", b, n_heads, t);
    return PIPO_ERR_ARG;
  }
  if (t >= kAttnDecodeMaxT) {
    set_error("attn_decode: %d keys, above the %d this kernel takes", t + 1, kAttnDecodeMaxT);
    return PIPO_ERR_UNSUPPORTED;
  }
  PIPO_TRY(check_heads("attn_decode", n_heads, n_kv_heads, head_dim));
  if (kv4 && ((int64_t)n_kv_heads * head_dim) % 256 != 0) {
    set_error("attn_decode: INT4 KV rows need a width %% 256 == 0 (%d)", n_kv_heads * head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  const int G = n_heads / n_kv_heads;
  const int HP = attn_decode_heads_per_wg(b, n_heads, n_kv_heads, kv4);
  const int T = t + 1;
  int S = attn_decode_splits(b, n_heads, n_kv_heads, t, kv4);
  if (!workspace || workspace_bytes < attn_decode_workspace_bytes(b, n_heads, head_dim, S)) S = 1;
  const int chunk = (T + S - 1) / S;
  S = (T + chunk - 1) / chunk;
  if (head_dim == 128)
    (kv4 ? launch_decode_d<128, true> : launch_decode_d<128, false>)(
        q, kc, vc, o, b, n_kv_heads, G, HP, t, S, chunk, workspace, st);
  else
    (kv4 ? launch_decode_d<64, true> : launch_decode_d<64, false>)(
        q, kc, vc, o, b, n_kv_heads, G, HP, t, S, chunk, workspace, st);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

pipo_status launch_attn_prefill(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                uint16_t* o, int b, int P, int n_heads, int n_kv_heads,
                                int head_dim, hipStream_t st) {
  if (b < 1 || n_heads < 1 || P < 1) {
    set_error("attn_prefill: bad shape b=%d P=%d heads=%d", b, P, n_heads);
    return PIPO_ERR_ARG;
  }
  PIPO_TRY(check_heads("attn_prefill", n_heads, n_kv_heads, head_dim));
  if ((int64_t)b * n_kv_heads * head_dim * kPK >= ((int64_t)1 << 31)) {
    set_error("attn_prefill: %d sequences of %d key/value heads of %d: a key block spans 2^31 "
              "elements or more", b, n_kv_heads, head_dim);
    return PIPO_ERR_UNSUPPORTED;
  }
  const dim3 grid((unsigned)((P + kPQ - 1) / kPQ), (unsigned)n_heads, (unsigned)b);
  if (head_dim == 128)
    launch(attn_prefill_k<128, kPrefillStages>, grid, dim3(256), 0, st, q, kc, vc, o, b, P,
           n_heads, n_kv_heads);
  else
    launch(attn_prefill_k<64, kPrefillStages>, grid, dim3(256), 0, st, q, kc, vc, o, b, P,
           n_heads, n_kv_heads);
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

}  // namespace pipo

// ---------------------------------------------------------------------------
// Decode attention for callers that cannot allocate (pipo_ops.h,
// pipo_op_attn_decode_noalloc): the split partials go to a fixed device
// array instead of a caller workspace.  In host code `scratch` names a
// host-side stand-in, so the array's device address is taken once per
// device with hipGetSymbolAddress and only that address is used.
namespace {

constexpr int64_t kScratchBytes = 4 << 20;
__device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

pipo_status scratch_address(void** out) {
  int dev = 0;
  PIPO_HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) {
    pipo::set_error("attn_decode_noalloc: device %d beyond %d", dev, kMaxDevices);
    return PIPO_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      pipo::set_error("attn_decode_noalloc: hipGetSymbolAddress failed (%s)",
                      hipGetErrorString(e));
      return PIPO_ERR_HIP;
    }
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return PIPO_OK;
}

}  // namespace

extern "C" pipo_status pipo_op_attn_decode_noalloc(const uint16_t* q, const uint16_t* kc,
                                                   const uint16_t* vc, uint16_t* o, int32_t b,
                                                   int32_t n_heads, int32_t head_dim, int32_t t,
                                                   void* stream) {
  pipo::clear_error();
  if (!q || !kc || !vc || !o) {
    pipo::set_error("attn_decode_noalloc: NULL pointer");
    return PIPO_ERR_ARG;
  }
  if (b < 1 || n_heads < 1 || t < 0 || head_dim < 1) {
    pipo::set_error("attn_decode_noalloc: bad shape b=%d heads=%d t=%d", b, n_heads, t);
    return PIPO_ERR_ARG;
  }
  const int64_t need = pipo::attn_decode_workspace_bytes(
      b, n_heads, head_dim, pipo::attn_decode_splits(b, n_heads, n_heads, t, false));
  if (need > kScratchBytes) {
    pipo::set_error("attn_decode_noalloc: the split partials need %lld bytes, above the %lld "
                    "bytes of the library's scratch array",
                    (long long)need, (long long)kScratchBytes);
    return PIPO_ERR_UNSUPPORTED;
  }
  void* ws = nullptr;
  if (need > 0) PIPO_TRY(scratch_address(&ws));
  return pipo::launch_attn_decode(q, kc, vc, o, b, n_heads, n_heads, head_dim, t, false,
                                  static_cast<float*>(ws), need,
                                  static_cast<hipStream_t>(stream));
}
