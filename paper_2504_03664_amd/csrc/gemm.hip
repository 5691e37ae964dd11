// Projection GEMMs of the decoder layer and the output head:
//   Y[M][N] = X[M][K] . W[N][K]^T  (+ bias, fused epilogue)
// with W in fp16 or group-wise INT4 (codes expanded to fp16 in registers,
// the paper's "compute directly on 4-bit weights", Section 3.4).
//
// The kernel is chosen by M (and N and the weight format):
//   * gemm_skinny (M <= 16, decode): every workgroup owns 16 or 64 rows of
//     W and all M rows of X; its waves split K; W streams from HBM straight
//     into MFMA operand registers (no LDS), X comes from L2.  Partial sums
//     are combined across waves in LDS in a fixed order.
//   * gemm_stream (16 < M <= 128, decode): waves split the rows of W, the
//     chunk of X that all of them need is staged once per workgroup in LDS,
//     and each wave keeps several chunks of its W rows in flight in
//     registers.  K may be split over workgroups; their fp32 partial sums
//     go to a workspace that gemm_combine adds up in a fixed order.
//   * gemm_tiled (M > 128, prefill with fewer big tiles): 128 x 128 output tiles, K staged
//     through double-buffered LDS in steps of 64, 4 waves of 64 x 64; tiles
//     ordered per XCD so that each XCD's L2 serves a compact block.
//   * gemm_big_f16 / gemm_big_w4 (prefill with at least 512 tiles of
//     256 x 256): 8 waves of 128 x 64 fed by global -> LDS loads (no
//     register staging) through rings of LDS stages; INT4 codes reach LDS
//     the same way and are expanded there, once per tile.
// The decode kernels read each weight once per pass and do so with
// non-temporal loads.
// All accumulate in fp32 with v_mfma_f32_16x16x32_f16, and INT4 codes
// become the same fp16 values (code * scale + min, rounded once) in every
// kernel.  The kernel, its configuration and the K split depend only on
// (M, N, K), so a given shape always sums in the same order; no workgroup
// reads another workgroup's results within a launch.
#include "common.h"
#include "device.h"

namespace pipo {

// Epilogue, split into what depends on the output row only (its offsets,
// computed once per row by kernels that own many columns of it) and the
// per-element part.  EPI_QKV: row m is sequence m / rows_per_seq at
// position pos0 + m % rows_per_seq, whose k and v go to cache row
// position * batch + sequence.
struct EpiRow {
  int64_t m;      // output row (>= M: none)
  int64_t off;    // m * ldo, or m * d for q (EPI_QKV)
  int64_t kvoff;  // EPI_QKV: cache row * dkv
};

template <int EPI>
__device__ __forceinline__ EpiRow epilogue_row(const GemmArgs& a, int64_t m) {
  EpiRow r{m, 0, 0};
  if (m >= a.M) return r;
  if constexpr (EPI == EPI_QKV) {
    // launch_gemm keeps M below 2^31, so 32-bit division is exact
    const uint32_t mm = (uint32_t)m, rps = (uint32_t)a.rows_per_seq;
    const uint32_t seq = mm / rps;
    const int64_t pos = a.pos0 + (int64_t)(mm - seq * rps);
    r.off = m * a.d;
    r.kvoff = (pos * a.batch + seq) * a.dkv;
  } else {
    r.off = m * a.ldo;
  }
  return r;
}

// bias of column n (0 past N or without bias)
__device__ __forceinline__ float epilogue_bias(const GemmArgs& a, int64_t n) {
  return (a.bias && n < a.N) ? h2f(a.bias[n]) : 0.f;
}

// v: the sum with the column's bias added
template <int EPI>
__device__ __forceinline__ void epilogue_store(const GemmArgs& a, const EpiRow& r, int64_t n,
                                               float v) {
  if (r.m >= a.M || n >= a.N) return;
  if constexpr (EPI == EPI_F16) {
    a.out16[r.off + n] = f2h(v);
  } else if constexpr (EPI == EPI_RELU_F16) {
    a.out16[r.off + n] = f2h(v > 0.f ? v : 0.f);
  } else if constexpr (EPI == EPI_ADD_F32) {
    a.out32[r.off + n] += v;
  } else if constexpr (EPI == EPI_F32) {
    a.out32[r.off + n] = v;
  } else {  // EPI_QKV
    if (n < a.d)
      a.q_out[r.off + n] = f2h(v * a.q_scale);
    else if (n < a.d + a.dkv)
      a.k_out[r.kvoff + (n - a.d)] = f2h(v);
    else
      a.v_out[r.kvoff + (n - a.d - a.dkv)] = f2h(v);
  }
}

template <int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int64_t m, int64_t n, float acc) {
  epilogue_store<EPI>(a, epilogue_row<EPI>(a, m), n, acc + epilogue_bias(a, n));
}

// ---------------------------------------------------------------------------
// skinny GEMM (decode)
//
// Workgroup = KW waves; it owns 16 NF rows of W (NF fragments) and all M
// (<= 16 MF) rows of X.  K is walked in 128-wide steps; wave w takes steps
// w, w + KW, ... UNR at a time so that UNR steps of W are in flight per
// lane.  In a step, lane (r, g) feeds four MFMAs (8 k each) with W row
// 16 f + r and X row 16 mf + r at the same k: fp16 W is read so that load i
// of the 16 lanes of a row covers 64 contiguous bytes (k = 32 i + 8 g), INT4
// codes as 32 consecutive k per lane (k = 32 g + 8 i).  Wave partials are
// added in LDS in wave order, then the epilogue runs.
template <int NF, int MF, int KW, int UNR, bool W4, bool PK>
struct SkinnyStep {
  u32x4 w[NF][4];  // fp16: four 8-half chunks; int4: w[f][0] holds 32 codes
  uint32_t sm[NF];
  h8 x[MF][4];

  __device__ __forceinline__ static int koff(int i, int g) { return W4 ? 32 * g + 8 * i : 32 * i + 8 * g; }

  // nb[f]: the first W row of fragment f
  __device__ __forceinline__ void load(const GemmArgs& a, const int64_t (&nb)[NF], int64_t s,
                                       int r, int g) {
    const int64_t K = a.K;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int64_t n = nb[f] + r;
      const bool ok = n < a.N;
      if constexpr (W4) {
        const int64_t kb = s * 128 + 32 * g;
        w[f][0] = ok ? load_u32x4_stream(a.Wq + w4_byte<PK>(n, kb, K))
                     : u32x4{0, 0, 0, 0};
        sm[f] = ok ? *reinterpret_cast<const uint32_t*>(a.Wsm + w4_sm<PK>(n, kb, K) * 2) : 0u;
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          w[f][i] = ok ? load_u32x4_stream(a.W + w16_index<PK>(n, s * 128 + koff(i, g), K))
                       : u32x4{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) {
      const int64_t m = 16 * mf + r;
      const uint16_t* p = a.X + m * K + s * 128;
#pragma unroll
      for (int i = 0; i < 4; ++i) x[mf][i] = m < a.M ? load_h8(p + koff(i, g)) : zero_h8();
    }
  }

  __device__ __forceinline__ void mma(f4 (&acc)[NF][MF]) const {
    // INT4: codes are expanded in the order (0, 4, 1, 5, ...) of each group
    // of eight k; X is permuted to match
    h8 xv[MF][4];
#pragma unroll
    for (int mf = 0; mf < MF; ++mf)
#pragma unroll
      for (int i = 0; i < 4; ++i) xv[mf][i] = W4 ? interleave_h8(x[mf][i]) : x[mf][i];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      h2 s2, m2;
      if constexpr (W4) scale_min_pairs(sm[f], s2, m2);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const h8 wv = W4 ? dequant8_interleaved(w[f][0][i], s2, m2) : __builtin_bit_cast(h8, w[f][i]);
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) acc[f][mf] = mfma16(wv, xv[mf][i], acc[f][mf]);
      }
    }
  }
};

template <int NF, int MF, int KW, int UNR, bool W4, int EPI, bool PK>
__global__ __launch_bounds__(KW * 64) void gemm_skinny(GemmArgs a) {
  __shared__ f4 red[KW][NF][MF][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  static_assert(EPI != EPI_SWIGLU || NF % 2 == 0, "SwiGLU pairs gate and up fragments");
  const int64_t n0 = (int64_t)blockIdx.x * (16 * NF);
  const int64_t nsteps = a.K / 128;
  // fragment f's first W row: 16 NF consecutive rows, or with EPI_SWIGLU the
  // gate rows h0 .. h0 + 8 NF - 1 and the up rows F + h0 .. (F = N / 2)
  const int64_t h0 = (int64_t)blockIdx.x * (8 * NF);
  int64_t nb[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    if constexpr (EPI == EPI_SWIGLU)
      nb[f] = f < NF / 2 ? h0 + 16 * f : a.N / 2 + h0 + 16 * (f - NF / 2);
    else
      nb[f] = n0 + 16 * f;
  }

  f4 acc[NF][MF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) acc[f][mf] = f4{0.f, 0.f, 0.f, 0.f};

  for (int64_t s = wave; s < nsteps; s += UNR * KW) {
    SkinnyStep<NF, MF, KW, UNR, W4, PK> st[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (s + u * KW < nsteps) st[u].load(a, nb, s + u * KW, r, g);
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (s + u * KW < nsteps) st[u].mma(acc);
  }

#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) red[wave][f][mf][lane] = acc[f][mf];
  __syncthreads();

  if constexpr (EPI == EPI_SWIGLU) {
    // element (f < NF / 2, mf, lane', j): output column h0 + 16 f + 4 (lane' / 16) + j
    // from the gate sum of fragment f and the up sum of fragment f + NF / 2,
    // each rounded to fp16 as a separate GEMM output would be
    constexpr int kElems = NF / 2 * MF * 64 * 4;
    const int64_t F = a.N / 2;
    for (int e = threadIdx.x; e < kElems; e += KW * 64) {
      const int j = e & 3, ln = (e >> 2) & 63, fm = e >> 8;
      const int f = fm / MF, mf = fm % MF;
      float gs = 0.f, us = 0.f;
#pragma unroll
      for (int w = 0; w < KW; ++w) {
        gs += red[w][f][mf][ln][j];
        us += red[w][f + NF / 2][mf][ln][j];
      }
      const int64_t m = 16 * mf + (ln & 15), i = h0 + 16 * f + 4 * (ln >> 4) + j;
      if (m < a.M && i < F) {
        const float gv = h2f(f2h(gs + 0.f)), uv = h2f(f2h(us + 0.f));
        a.out16[m * a.ldo + i] = f2h(gv / (1.f + expf(-gv)) * uv);
      }
    }
  } else {
    // element (f, mf, lane', j): W row n0 + 16 f + 4 (lane' / 16) + j, X row 16 mf + lane' % 16
    constexpr int kElems = NF * MF * 64 * 4;
    for (int e = threadIdx.x; e < kElems; e += KW * 64) {
      const int j = e & 3, ln = (e >> 2) & 63, fm = e >> 8;
      const int f = fm / MF, mf = fm % MF;
      float sum = 0.f;
#pragma unroll
      for (int w = 0; w < KW; ++w) sum += red[w][f][mf][ln][j];
      epilogue<EPI>(a, 16 * mf + (ln & 15), n0 + 16 * f + 4 * (ln >> 4) + j, sum);
    }
  }
}

// ---------------------------------------------------------------------------
// streaming GEMM (decode at 16 < M <= 128)
//
// Workgroup = KW waves; wave w owns W rows n0 + 16 NF w .. + 16 NF and the
// workgroup covers k in [z kper, (z + 1) kper), z = blockIdx.y.  K is walked
// in chunks of KC: the X chunk (16 MF rows x KC) is loaded once per
// workgroup, PD chunks ahead into registers and then into one of two LDS
// buffers, one barrier per chunk; each wave holds PD chunks of its W rows
// in registers, refilling a chunk's registers as soon as its MFMAs are
// issued.  (With X loaded only one chunk ahead, every chunk waited for an
// L2 round trip before its barrier.)  Every load is unconditional (row and
// chunk indexes are clamped: rows past M or N are computed and never
// stored, a clamped chunk is loaded again and not used), which keeps the
// compiler's wait counts exact so that the prefetch really stays in flight.
// In a chunk, lane (r, g) feeds MFMA i with W row 16 f + r at
// k = 32 i + 8 g (fp16) or k = 32 g + 8 i (INT4: 32 consecutive codes per
// lane, expanded in interleaved order, X permuted to match).
template <int NF, int MF, int KW, int PD, bool W4, int KC>
struct StreamCfg {
  static constexpr int kXRows = 16 * MF;
  static constexpr int kXLd = KC + 8;  // halves per LDS row (padding against bank conflicts)
  static constexpr int kThreads = KW * 64;
  static constexpr int kXH8 = kXRows * KC / 8;                       // 8-half pieces per X chunk
  static constexpr int kXPerThread = (kXH8 + kThreads - 1) / kThreads;
  static constexpr int kWRegs = W4 ? KC / 128 : KC / 32;             // u32x4 per W row per chunk
  static constexpr int kRowsPerWG = 16 * NF * KW;
};

__device__ __forceinline__ int64_t clamp_hi(int64_t v, int64_t hi) { return v < hi ? v : hi; }

template <int NF, int MF, int KW, int PD, bool W4, int KC, int EPI, bool PK>
__global__ __launch_bounds__(KW * 64) void gemm_stream(GemmArgs a, float* part, int64_t kper) {
  using C = StreamCfg<NF, MF, KW, PD, W4, KC>;
  __shared__ __attribute__((aligned(16))) uint16_t Xs[2][C::kXRows * C::kXLd];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, g = lane >> 4;
  const int64_t nw0 = ((int64_t)blockIdx.x * KW + wave) * (16 * NF);
  const int64_t kbeg = (int64_t)blockIdx.y * kper;
  const int64_t nch = kper / KC;
  const int64_t K = a.K;
  int64_t wrow[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) wrow[f] = clamp_hi(nw0 + 16 * f + r, a.N - 1);

  struct WChunk {
    u32x4 w[NF][C::kWRegs];
    uint32_t sm[NF][W4 ? KC / 128 : 1];
  };
  // Fragment order: a lane's 16 bytes of a 16-row block sit at the same
  // offset in every block of its row group, and the blocks of a row group
  // follow each other along k, so a lane's address is its own base plus a
  // workgroup-uniform block offset (fp16: 32-k blocks of 1 KiB; INT4:
  // 128-k blocks of 1 KiB of codes and 32 (scale, min) words).
  const uint8_t* wlane[NF];
  const uint32_t* smlane[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int64_t grp = wrow[f] >> 4;
    if constexpr (W4) {
      wlane[f] = a.Wq + grp * (K >> 7) * 1024 + (((wrow[f] & 15) + 16 * g) << 4);
      smlane[f] = reinterpret_cast<const uint32_t*>(a.Wsm) + grp * (K >> 7) * 32 +
                  (wrow[f] & 15) * 2 + (g >> 1);
    } else {
      wlane[f] = reinterpret_cast<const uint8_t*>(a.W) + grp * (K >> 5) * 1024 +
                 (((wrow[f] & 15) + 16 * g) << 4);
      smlane[f] = nullptr;
    }
  }
  const auto load_w = [&](WChunk& F, int64_t c) {
    const int64_t k0 = kbeg + clamp_hi(c, nch - 1) * KC;
    if constexpr (PK) {
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        if constexpr (W4) {
#pragma unroll
          for (int t = 0; t < KC / 128; ++t) {
            const int64_t blk = (k0 >> 7) + t;
            F.w[f][t] = load_u32x4_stream(wlane[f] + blk * 1024);
            F.sm[f][t] = smlane[f][blk * 32];
          }
        } else {
#pragma unroll
          for (int i = 0; i < C::kWRegs; ++i)
            F.w[f][i] = load_u32x4_stream(wlane[f] + ((k0 >> 5) + i) * 1024);
        }
      }
      return;
    }
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      if constexpr (W4) {
#pragma unroll
        for (int t = 0; t < KC / 128; ++t) {
          const int64_t kb = k0 + 128 * t + 32 * g;
          F.w[f][t] = load_u32x4_stream(a.Wq + w4_byte<PK>(wrow[f], kb, K));
          F.sm[f][t] = *reinterpret_cast<const uint32_t*>(a.Wsm + w4_sm<PK>(wrow[f], kb, K) * 2);
        }
      } else {
#pragma unroll
        for (int i = 0; i < C::kWRegs; ++i)
          F.w[f][i] = load_u32x4_stream(a.W + w16_index<PK>(wrow[f], k0 + 32 * i + 8 * g, K));
      }
    }
  };
  // X chunks travel through registers PD chunks ahead of their use, like W:
  // chunk c sits in ring slot c % PD from its load (iteration c - 1 - PD)
  // until it is stored to LDS (end of iteration c - 1)
  h8 xr[PD][C::kXPerThread];
  const auto load_x = [&](int slot, int64_t c) {
    const int64_t k0 = kbeg + clamp_hi(c, nch - 1) * KC;
#pragma unroll
    for (int j = 0; j < C::kXPerThread; ++j) {
      const int e = tid + j * C::kThreads < C::kXH8 ? tid + j * C::kThreads : C::kXH8 - 1;
      const int row = e / (KC / 8), col = (e % (KC / 8)) * 8;
      xr[slot][j] = load_h8(a.X + clamp_hi(row, a.M - 1) * K + k0 + col);
    }
  };
  // INT4: X is stored already permuted to the codes' interleaved order
  // (once per workgroup rather than once per wave and use)
  const auto store_x = [&](int b, int slot) {
#pragma unroll
    for (int j = 0; j < C::kXPerThread; ++j) {
      const int e = tid + j * C::kThreads;
      if (e < C::kXH8) {
        const int row = e / (KC / 8), col = (e % (KC / 8)) * 8;
        *reinterpret_cast<h8*>(&Xs[b][row * C::kXLd + col]) =
            W4 ? interleave_h8(xr[slot][j]) : xr[slot][j];
      }
    }
  };
  f4 acc[NF][MF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) acc[f][mf] = f4{0.f, 0.f, 0.f, 0.f};
  const auto compute = [&](const WChunk& F, int b) {
#pragma unroll
    for (int t = 0; t < KC / 128; ++t) {
      h2 s2[NF], m2[NF];
      if constexpr (W4) {
#pragma unroll
        for (int f = 0; f < NF; ++f) scale_min_pairs(F.sm[f][t], s2[f], m2[f]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kl = 128 * t + (W4 ? 32 * g + 8 * i : 32 * i + 8 * g);
        h8 xv[MF];
#pragma unroll
        for (int mf = 0; mf < MF; ++mf)
          xv[mf] = *reinterpret_cast<const h8*>(&Xs[b][(16 * mf + r) * C::kXLd + kl]);
#pragma unroll
        for (int f = 0; f < NF; ++f) {
          const h8 wv = W4 ? dequant8_interleaved(F.w[f][t][i], s2[f], m2[f])
                           : __builtin_bit_cast(h8, F.w[f][4 * t + i]);
#pragma unroll
          for (int mf = 0; mf < MF; ++mf) acc[f][mf] = mfma16(wv, xv[mf], acc[f][mf]);
        }
      }
    }
  };

  WChunk F[PD];
  load_x(0, 0);
  store_x(0, 0);
#pragma unroll
  for (int p = 1; p <= PD; ++p) load_x(p % PD, p);
#pragma unroll
  for (int p = 0; p < PD; ++p) {
    load_w(F[p], p);
    __builtin_amdgcn_sched_barrier(0);  // keep the chunks' loads in chunk order
  }
  __syncthreads();
  for (int64_t c0 = 0; c0 < nch; c0 += PD) {
#pragma unroll
    for (int p = 0; p < PD; ++p) {
      const int64_t c = c0 + p;
      if (c < nch) compute(F[p], (int)(c & 1));
      load_w(F[p], c + PD);
      __builtin_amdgcn_sched_barrier(0);
      // buffer (c + 1) & 1 was last read in chunk c - 1, before the barrier
      store_x((int)((c + 1) & 1), (p + 1) % PD);
      load_x((p + 1) % PD, c + 1 + PD);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
    }
  }

  // acc[f][mf] element j: W row nw0 + 16 f + 4 g + j, X row 16 mf + r
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t m = 16 * mf + r, n = nw0 + 16 * f + 4 * g + j;
        if (gridDim.y == 1) {
          epilogue<EPI>(a, m, n, acc[f][mf][j]);
        } else if (m < a.M && n < a.N) {
          part[((int64_t)blockIdx.y * a.M + m) * a.N + n] = acc[f][mf][j];
        }
      }
}

// out = sum over z = 0 .. S-1 (in that order, from 0) of part[z], then the
// epilogue.  A thread takes V adjacent columns of one row (V = 4 when N is a
// multiple of 4 and the partials are 16-byte aligned) and issues the loads
// of all S partials before the first add; M * N < 2^31 (checked by the host).
template <int EPI, int S, int V>
__global__ __launch_bounds__(256) void gemm_combine(GemmArgs a, const float* __restrict__ part) {
  const int NV = (int)(a.N / V);
  const int q = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (q >= (int)a.M * NV) return;
  const int m = q / NV, n = (q - m * NV) * V;
  const int64_t MN = a.M * a.N;
  const float* p = part + (int64_t)m * a.N + n;
  float v[S][V];
#pragma unroll
  for (int z = 0; z < S; ++z) {
    if constexpr (V == 4) {
      const f4 t = *reinterpret_cast<const f4*>(p + z * MN);
#pragma unroll
      for (int j = 0; j < 4; ++j) v[z][j] = t[j];
    } else {
      v[z][0] = p[z * MN];
    }
  }
  const EpiRow row = epilogue_row<EPI>(a, m);
#pragma unroll
  for (int j = 0; j < V; ++j) {
    float sum = 0.f;
#pragma unroll
    for (int z = 0; z < S; ++z) sum += v[z][j];
    epilogue_store<EPI>(a, row, n + j, sum + epilogue_bias(a, n + j));
  }
}

template <int EPI, int V>
static void launch_combine_v(const GemmArgs& a, const float* ws, int S, hipStream_t st) {
  const dim3 grid((unsigned)((a.M * (a.N / V) + 255) / 256));
  switch (S) {
    case 2: launch((gemm_combine<EPI, 2, V>), grid, dim3(256), 0, st, a, ws); break;
    case 4: launch((gemm_combine<EPI, 4, V>), grid, dim3(256), 0, st, a, ws); break;
    default: launch((gemm_combine<EPI, 8, V>), grid, dim3(256), 0, st, a, ws); break;
  }
}

template <int EPI>
static void launch_combine(const GemmArgs& a, const float* ws, int S, hipStream_t st) {
  if (a.N % 4 == 0 && reinterpret_cast<uintptr_t>(ws) % 16 == 0)
    launch_combine_v<EPI, 4>(a, ws, S, st);
  else
    launch_combine_v<EPI, 1>(a, ws, S, st);
}

// ---------------------------------------------------------------------------
// tiled GEMM (prefill)
constexpr int kTBM = 128, kTBN = 128, kTBK = 64, kTPad = 8;
constexpr int kTThreads = 256;  // 2 x 2 waves of 64 x 64
constexpr int kXcds = 8;        // accelerator complex dies of an MI355X, each with its own L2
constexpr int kTGroupM = 4;

template <bool W4, int EPI, bool PK>
__global__ __launch_bounds__(kTThreads) void gemm_tiled(GemmArgs a) {
  constexpr int LDS_ROW = kTBK + kTPad;  // halves
  __shared__ __attribute__((aligned(16))) uint16_t As[2][kTBM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][kTBN * LDS_ROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  // Tile order.  Workgroups are dealt to the 8 XCDs round-robin, and each
  // XCD has its own L2: give XCD x a contiguous range of tiles, and walk
  // that range in groups of kTGroupM row tiles (row tile fastest), so that
  // the workgroups an XCD runs at once share A rows and B columns in L2.
  const int64_t tiles_m = (a.M + kTBM - 1) / kTBM, tiles_n = (a.N + kTBN - 1) / kTBN;
  const int64_t total = tiles_m * tiles_n;
  const int64_t per_xcd = (total + kXcds - 1) / kXcds;
  const int64_t tile = (int64_t)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (tile >= total) return;
  const int64_t group = tile / (kTGroupM * tiles_n);
  const int64_t first_m = group * kTGroupM;
  const int64_t gm = tiles_m - first_m < kTGroupM ? tiles_m - first_m : kTGroupM;
  const int64_t in_group = tile - group * kTGroupM * tiles_n;
  const int64_t m0 = (first_m + in_group % gm) * kTBM;
  const int64_t n0 = (in_group / gm) * kTBN;
  const int64_t K = a.K;
  const int64_t KT = K / kTBK;

  // global -> register staging: A and fp16 B take 4 chunks of 8 halves per
  // thread (row = c / 8, col = 8 (c % 8)); INT4 B takes one 32-code chunk.
  // With B in fragment order a wave's 64 chunks are one 16-row x 32-k
  // block (1 KiB contiguous; INT4: 32 threads read a 512-byte half block).
  const auto b_row = [](int c) { return PK ? ((c >> 7) << 4) + (c & 15) : c >> 3; };
  const auto b_col = [](int c) { return PK ? ((c >> 6) & 1) * 32 + ((c >> 4) & 3) * 8 : (c & 7) * 8; };
  const auto b_row_w4 = [](int t, int64_t) { return PK ? ((t >> 5) << 4) + (t & 15) : t >> 1; };
  const auto b_half_w4 = [](int t, int64_t) { return PK ? (t >> 4) & 1 : t & 1; };
  h8 ra[4], rb[4];
  const auto load_tile = [&](int64_t kt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + i * kTThreads;
      const int row = c >> 3, col = (c & 7) * 8;
      const int64_t m = m0 + row;
      ra[i] = m < a.M ? load_h8(a.X + m * K + kt * kTBK + col) : zero_h8();
    }
    if constexpr (W4) {
      const int row = b_row_w4(tid, kt), half = b_half_w4(tid, kt);
      const int64_t n = n0 + row;
      if (n < a.N) {
        const int64_t kc = kt * kTBK + half * 32;
        const u32x4 codes = *reinterpret_cast<const u32x4*>(a.Wq + w4_byte<PK>(n, kc, K));
        const uint32_t smw = *reinterpret_cast<const uint32_t*>(a.Wsm + w4_sm<PK>(n, kc, K) * 2);
        h2 s2, m2;
        scale_min_pairs(smw, s2, m2);
#pragma unroll
        for (int i = 0; i < 4; ++i) rb[i] = dequant8(codes[i], s2, m2);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) rb[i] = zero_h8();
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + i * kTThreads;
        const int row = b_row(c), col = b_col(c);
        const int64_t n = n0 + row;
        rb[i] = n < a.N ? load_h8(a.W + w16_index<PK>(n, kt * kTBK + col, K)) : zero_h8();
      }
    }
  };
  const auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + i * kTThreads;
      const int row = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<h8*>(&As[buf][row * LDS_ROW + col]) = ra[i];
    }
    if constexpr (W4) {
      const int row = b_row_w4(tid, 0), half = b_half_w4(tid, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<h8*>(&Bs[buf][row * LDS_ROW + half * 32 + 8 * i]) = rb[i];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + i * kTThreads;
        *reinterpret_cast<h8*>(&Bs[buf][b_row(c) * LDS_ROW + b_col(c)]) = rb[i];
      }
    }
  };

  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int64_t kt = 0; kt < KT; ++kt) {
    const int buf = (int)(kt & 1);
    if (kt + 1 < KT) load_tile(kt + 1);
#pragma unroll
    for (int ks = 0; ks < kTBK / 32; ++ks) {
      h8 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const h8*>(
            &As[buf][(wm * 64 + i * 16 + r) * LDS_ROW + ks * 32 + g * 8]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bf[j] = *reinterpret_cast<const h8*>(
            &Bs[buf][(wn * 64 + j * 16 + r) * LDS_ROW + ks * 32 + g * 8]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16(af[i], bf[j], acc[i][j]);
    }
    if (kt + 1 < KT) store_tile(buf ^ 1);
    __syncthreads();
  }

  // acc[i][j] element e: row m0 + 64 wm + 16 i + 4 g + e, col n0 + 64 wn + 16 j + r;
  // biases once per column, row offsets once per row
  float bias[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) bias[j] = epilogue_bias(a, n0 + wn * 64 + j * 16 + r);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const EpiRow row = epilogue_row<EPI>(a, m0 + wm * 64 + i * 16 + 4 * g + e);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        epilogue_store<EPI>(a, row, n0 + wn * 64 + j * 16 + r, acc[i][j][e] + bias[j]);
    }
}

// ---------------------------------------------------------------------------
// big-tile GEMMs (prefill with at least kBigMinTiles 256 x 256 tiles, enough
// to fill the chip twice over): each W element read into LDS feeds 256 rows
// of X instead of 128, and each LDS operand read feeds more MFMAs.  Same
// tile order as gemm_tiled; the same MFMA per 32-wide k block in the same k
// order, so for a given K every kernel gives the same bits.
// ---------------------------------------------------------------------------
constexpr int64_t kBigMinTiles = 512;

__host__ __device__ constexpr int64_t big_tiles(int64_t M, int64_t N) {
  return ((M + 255) / 256) * ((N + 255) / 256);
}

constexpr int kBM = 256, kBN = 256;

// fp16 W (fragment order, or row-major: PK): 8 waves (two per SIMD) of 128 x 64 (8 x 4
// accumulator fragments), K in stages of 32.  Everything moves from global
// memory straight into LDS by the load unit (global_load_lds_dwordx4: lane
// l of a wave writes bytes 16 l .. 16 l + 15 of its destination).  A W
// stage is 16 row blocks of 16 rows x 32 k = 1 KiB in MFMA operand order
// (lane slot r + 16 g holds row r, k = 8 g .. 8 g + 7), in a ring of four
// stages; fragment reads are one contiguous KiB per wave.  X moves 64 k at
// a time: each load covers 8 rows x 128 bytes, whole cache lines of the
// row-major activations (loads of 16 rows x 64 bytes fetched every line
// twice, once per 32-k stage), into a ring of three 32 KiB slots where row
// r of a 16-row block keeps its 16-byte chunk c at position c ^ ((r / 2) %
// 8), which leaves the fragment reads free of bank conflicts (160 KiB of
// LDS in all).  Stage t is read while the next two are in flight and the
// loads of stage t + 3 (W) and of half a 64-k X stage are issued into
// buffers already read.  Fragment registers are double-buffered: the reads
// of stage t are spread over the MFMAs of stage t - 1.  Rows past M (and
// row blocks past N) are loaded from the last valid row and their results
// dropped.
constexpr int kFThreads = 512;
constexpr int kFStages = 4;              // LDS stages of the INT4 kernel's ring

template <int EPI, bool PK>
__global__ __launch_bounds__(kFThreads) void gemm_big_f16(GemmArgs a) {
  constexpr int FM = 8, FN = 4;  // fragments per wave
  constexpr int BPW = 2;         // W row blocks each wave moves per stage
  constexpr int PER_STAGE = 2 * BPW;
  constexpr int XSLOT = 32 * 1024, XSLOTS = 3, WSLOT = 16 * 1024, WSLOTS = 4;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[XSLOTS * XSLOT + WSLOTS * WSLOT];
  uint8_t* const xring = lds;
  uint8_t* const wring = lds + XSLOTS * XSLOT;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int64_t tiles_m = (a.M + kBM - 1) / kBM, tiles_n = (a.N + kBN - 1) / kBN;
  const int64_t total = tiles_m * tiles_n;
  const int64_t per_xcd = (total + kXcds - 1) / kXcds;
  const int64_t tile = (int64_t)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (tile >= total) return;
  const int64_t group = tile / (kTGroupM * tiles_n);
  const int64_t first_m = group * kTGroupM;
  const int64_t gm = tiles_m - first_m < kTGroupM ? tiles_m - first_m : kTGroupM;
  const int64_t in_group = tile - group * kTGroupM * tiles_n;
  const int64_t m0 = (first_m + in_group % gm) * kBM;
  const int64_t n0 = (in_group / gm) * kBN;
  const int64_t K = a.K;
  const int KT = (int)(K / 32);
  const int KS = KT / 2;         // 64-wide X stages

  const int r = lane & 15, g = lane >> 4;
  // X: wave w moves row blocks 2w and 2w + 1, half q (rows 8q .. 8q + 7)
  // of a 64-k stage per step; lane l takes row 8q + l / 8 and chunk
  // (l % 8) ^ ((row >> 1) & 7) of the row's 128 bytes
  const uint16_t* xsrc[2][2];
#pragma unroll
  for (int bb = 0; bb < 2; ++bb)
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int row = 8 * q + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      int64_t m = m0 + 16 * (2 * wave + bb) + row;
      m = m < a.M ? m : a.M - 1;
      xsrc[bb][q] = a.X + m * K + 8 * c;
    }
  const uint16_t* bsrc[BPW];
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    if constexpr (PK) {
      int64_t nb = (n0 >> 4) + BPW * wave + i;
      nb = nb < (a.N >> 4) ? nb : (a.N >> 4) - 1;
      bsrc[i] = a.W + nb * (K >> 5) * 512 + lane * 8;
    } else {
      int64_t n = n0 + 16 * (BPW * wave + i) + r;
      n = n < a.N ? n : a.N - 1;
      bsrc[i] = a.W + n * K + 8 * g;
    }
  }
  constexpr int kBStep = PK ? 512 : 32;
  // step u issues W stage u + 3 and half u & 1 of X stage (u >> 1) + 2
  // (arithmetic shift: u = -4 .. -1 are the prologue)
  const auto issue = [&](int u) {
    if (u >= -3) {
      const int ws = u + 3 < KT ? u + 3 : KT - 1;
      uint8_t* st = wring + ((u + 3) % WSLOTS) * WSLOT;
#pragma unroll
      for (int i = 0; i < BPW; ++i)
        lds_dma16(bsrc[i] + ws * kBStep, st + (BPW * wave + i) * 1024);
    }
    const int s = (u >> 1) + 2, q = u & 1;
    const int sc = s < KS ? s : KS - 1;
    uint8_t* xs = xring + (s % XSLOTS) * XSLOT;
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
      lds_dma16(xsrc[bb][q] + sc * 64, xs + (2 * wave + bb) * 2048 + q * 1024);
  };
  const auto read = [&](int t, h8 (&fa)[FM], h8 (&fb)[FN]) {
    const uint8_t* ws = wring + (t % WSLOTS) * WSLOT;
#pragma unroll
    for (int j = 0; j < FN; ++j)
      fb[j] = *reinterpret_cast<const h8*>(ws + (FN * wn + j) * 1024 + lane * 16);
    const uint8_t* xs = xring + ((t >> 1) % XSLOTS) * XSLOT;
    const int c = (g + 4 * (t & 1)) ^ ((r >> 1) & 7);
    const int off = (r >> 3) * 1024 + (r & 7) * 128 + 16 * c;
#pragma unroll
    for (int i = 0; i < FM; ++i)
      fa[i] = *reinterpret_cast<const h8*>(xs + (FM * wm + i) * 2048 + off);
  };
  f4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  const auto mma = [&](const h8 (&fa)[FM], const h8 (&fb)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = mfma16(fa[i], fb[j], acc[i][j]);
  };
  h8 fa0[FM], fb0[FN], fa1[FM], fb1[FN];
  const auto step = [&](int t, h8 (&ra)[FM], h8 (&rb)[FN], h8 (&ca)[FM], h8 (&cb)[FN]) {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(2 * PER_STAGE, true));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue(t);
    read(t, ra, rb);
    mma(ca, cb);
#pragma unroll
    for (int k = 0; k < PER_STAGE; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // global -> LDS load
    }
#pragma unroll
    for (int k = 0; k < FM + FN; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMA
    }
    __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - 2 * PER_STAGE - 2 * (FM + FN), 0);
  };
  issue(-4);  // X stage 0, rows 0-7 of each block (no W)
  issue(-3);
  issue(-2);
  issue(-1);
  // W stage 0 and both halves of X stage 0 landed (steps -2, -1 may be in flight)
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(2 * PER_STAGE, true));
  __builtin_amdgcn_s_barrier();
  issue(0);
  read(0, fa0, fb0);
  int t = 1;
  for (; t < KT - 1; t += 2) {
    step(t, fa1, fb1, fa0, fb0);
    step(t + 1, fa0, fb0, fa1, fb1);
  }
  step(t, fa1, fb1, fa0, fb0);
  // every load landed (none may write LDS after the workgroup ends)
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, true));
  mma(fa1, fb1);

  // acc[i][j] element e: row m0 + 128 wm + 16 i + 4 g + e, col n0 + 64 wn + 16 j + r
  float bias[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) bias[j] = epilogue_bias(a, n0 + wn * 64 + j * 16 + r);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const EpiRow row = epilogue_row<EPI>(a, m0 + wm * 128 + i * 16 + 4 * g + e);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        epilogue_store<EPI>(a, row, n0 + wn * 64 + j * 16 + r, acc[i][j][e] + bias[j]);
    }
}

// INT4 W (fragment order or row-major): as gemm_big_f16, with the W area of
// a stage filled by the threads.  The codes (16 bytes per W row and stage)
// and (scale, min) pairs of a stage reach LDS through the load unit one
// stage ahead of X; at step t every thread expands 16 codes of stage t + 1
// (W row tid / 2, k 16 (tid & 1) .. + 15) into two 16-byte fragment slots,
// so each code is expanded once per 256 rows of X.  A stage is X 16 KiB,
// expanded W 16 KiB, codes 4 KiB, pairs 1 KiB; four stages, 148 KiB.
template <int EPI, bool PK>
__global__ __launch_bounds__(kFThreads) void gemm_big_w4(GemmArgs a) {
  constexpr int FM = 8, FN = 4;
  constexpr int BPW = 2;
  constexpr int PER_STEP = BPW + 1;               // X blocks + one code or pair load
  constexpr int STAGE = 32 * 1024 + 4096 + 1024;  // bytes per LDS stage
  constexpr int WOFF = 16 * 1024, COFF = 32 * 1024, SOFF = 36 * 1024;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kFStages * STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int64_t tiles_m = (a.M + kBM - 1) / kBM, tiles_n = (a.N + kBN - 1) / kBN;
  const int64_t total = tiles_m * tiles_n;
  const int64_t per_xcd = (total + kXcds - 1) / kXcds;
  const int64_t tile = (int64_t)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (tile >= total) return;
  const int64_t group = tile / (kTGroupM * tiles_n);
  const int64_t first_m = group * kTGroupM;
  const int64_t gm = tiles_m - first_m < kTGroupM ? tiles_m - first_m : kTGroupM;
  const int64_t in_group = tile - group * kTGroupM * tiles_n;
  const int64_t m0 = (first_m + in_group % gm) * kBM;
  const int64_t n0 = (in_group / gm) * kBN;
  const int64_t K = a.K;
  const int KT = (int)(K / 32);

  const int r = lane & 15, g = lane >> 4;
  const uint16_t* asrc[BPW];
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    int64_t m = m0 + 16 * (BPW * wave + i) + r;
    m = m < a.M ? m : a.M - 1;
    asrc[i] = a.X + m * K + 8 * g;
  }
  // waves 0-3: the codes of W rows 64 w + lane; waves 4-7: their pairs
  int64_t wn_row = n0 + 64 * (wave & 3) + lane;
  wn_row = wn_row < a.N ? wn_row : a.N - 1;
  const auto issue_x = [&](int src, int buf) {
    uint8_t* st = lds + (buf % kFStages) * STAGE;
#pragma unroll
    for (int i = 0; i < BPW; ++i) lds_dma16(asrc[i] + src * 32, st + (BPW * wave + i) * 1024);
  };
  const auto issue_w = [&](int src, int buf) {
    uint8_t* st = lds + (buf % kFStages) * STAGE;
    if (wave < 4)
      lds_dma16(a.Wq + w4_byte<PK>(wn_row, 32 * src, K), st + COFF + 64 * wave * 16);
    else
      __builtin_amdgcn_global_load_lds(a.Wsm + w4_sm<PK>(wn_row, 32 * src, K) * 2,
                                       (__attribute__((address_space(3))) void*)(st + SOFF + 64 * (wave - 4) * 4),
                                       4, 0, 0);
  };
  // thread: W row tid / 2 of the tile, k 16 (tid & 1) .. + 15 of the stage
  const auto expand = [&](int buf) {
    uint8_t* st = lds + (buf % kFStages) * STAGE;
    const int row = tid >> 1, half = tid & 1;
    const u32x2 c = *reinterpret_cast<const u32x2*>(st + COFF + row * 16 + half * 8);
    const uint32_t sm = *reinterpret_cast<const uint32_t*>(st + SOFF + row * 4);
    h2 s2, m2;
    scale_min_pairs(sm, s2, m2);
    uint8_t* wb = st + WOFF + (row >> 4) * 1024 + ((row & 15) + 32 * half) * 16;
    *reinterpret_cast<h8*>(wb) = dequant8(c[0], s2, m2);
    *reinterpret_cast<h8*>(wb + 256) = dequant8(c[1], s2, m2);
  };
  const auto read = [&](int t, h8 (&fa)[FM], h8 (&fb)[FN]) {
    const uint8_t* st = lds + (t % kFStages) * STAGE;
#pragma unroll
    for (int j = 0; j < FN; ++j)
      fb[j] = *reinterpret_cast<const h8*>(st + WOFF + (FN * wn + j) * 1024 + lane * 16);
#pragma unroll
    for (int i = 0; i < FM; ++i)
      fa[i] = *reinterpret_cast<const h8*>(st + (FM * wm + i) * 1024 + lane * 16);
  };
  f4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  const auto mma = [&](const h8 (&fa)[FM], const h8 (&fb)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = mfma16(fa[i], fb[j], acc[i][j]);
  };
  const auto clampk = [&](int s) { return s < KT ? s : KT - 1; };
  // step t: codes of stage t + 1 and X of stage t landed; codes of t + 4
  // and X of t + 3 issued; codes of t + 1 expanded; stage t read while the
  // MFMAs of t - 1 run
  h8 fa0[FM], fb0[FN], fa1[FM], fb1[FN];
  const auto step = [&](int t, h8 (&ra)[FM], h8 (&rb)[FN], h8 (&ca)[FM], h8 (&cb)[FN], bool mm) {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(2 * PER_STEP, true));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue_w(clampk(t + 4), t + 4);
    issue_x(clampk(t + 3), t + 3);
    expand(t + 1);
    read(t, ra, rb);
    if (mm) mma(ca, cb);
    // two MFMAs before the loads, so that the MFMA pipe restarts right
    // after the barrier; then one fragment read and two MFMAs, in turn
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, PER_STEP, 0);
#pragma unroll
    for (int k = 0; k < FM + FN; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - 2 - 2 * (FM + FN), 0);
  };
  issue_w(0, 0);
  issue_w(1, 1);
  issue_x(0, 0);
  issue_w(2, 2);
  issue_x(1, 1);
  issue_w(3, 3);
  issue_x(2, 2);
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(2 * PER_STEP + 2, true));  // codes of stage 0
  __builtin_amdgcn_s_barrier();
  expand(0);
  step(0, fa0, fb0, fa1, fb1, false);
  int t = 1;
  for (; t < KT - 1; t += 2) {
    step(t, fa1, fb1, fa0, fb0, true);
    step(t + 1, fa0, fb0, fa1, fb1, true);
  }
  step(t, fa1, fb1, fa0, fb0, true);
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, true));
  mma(fa1, fb1);

  float bias[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) bias[j] = epilogue_bias(a, n0 + wn * 64 + j * 16 + r);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const EpiRow row = epilogue_row<EPI>(a, m0 + wm * 128 + i * 16 + 4 * g + e);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        epilogue_store<EPI>(a, row, n0 + wn * 64 + j * 16 + r, acc[i][j][e] + bias[j]);
    }
}

// ---------------------------------------------------------------------------
// skinny configurations by M: (waves, steps in flight per wave)
// ---------------------------------------------------------------------------
template <int MF> struct SkinnyCfg;
template <> struct SkinnyCfg<1> { static constexpr int KW = 8, UNR = 2; };

template <int NF, bool W4, int EPI, bool PK>
static void launch_skinny(const GemmArgs& a, hipStream_t st) {
  using C = SkinnyCfg<1>;
  const dim3 grid((unsigned)((a.N + 16 * NF - 1) / (16 * NF)));
  launch((gemm_skinny<NF, 1, C::KW, C::UNR, W4, EPI, PK>), grid, dim3(C::KW * 64), 0, st, a);
}

// streaming configurations by (W format, 16-row blocks of X): rows per
// wave (16 NF), waves, chunks in flight, chunk length; and a fallback with
// 128-k chunks for K that the chunk length does not divide
template <bool W4, int MF> struct StreamSel;
template <> struct StreamSel<false, 2> { static constexpr int NF = 1, KW = 8, PD = 2, KC = 128; };
template <> struct StreamSel<false, 4> { static constexpr int NF = 1, KW = 8, PD = 2, KC = 128; };
template <> struct StreamSel<false, 8> { static constexpr int NF = 1, KW = 8, PD = 2, KC = 128; };
template <> struct StreamSel<true, 2> { static constexpr int NF = 1, KW = 8, PD = 2, KC = 256; };
template <> struct StreamSel<true, 4> { static constexpr int NF = 2, KW = 8, PD = 4, KC = 256; };
template <> struct StreamSel<true, 8> { static constexpr int NF = 2, KW = 8, PD = 4, KC = 128; };
template <bool W4, int MF> struct StreamFallback {
  static constexpr int NF = StreamSel<W4, MF>::NF, KW = StreamSel<W4, MF>::KW;
  static constexpr int PD = StreamSel<W4, MF>::KC == 128 ? StreamSel<W4, MF>::PD : 2 * StreamSel<W4, MF>::PD;
  static constexpr int KC = 128;
};

constexpr int kStreamMaxM = 128;
constexpr int kStreamMaxSplits = 8;
constexpr int64_t kStreamMaxWGs = 256;  // about one workgroup per CU measured best

static int stream_mf(int64_t M) { return M <= 32 ? 2 : (M <= 64 ? 4 : 8); }

// K split: the largest power of two (up to the cap) that keeps the grid
// within kStreamMaxWGs workgroups and the split a multiple of the chunk
static int stream_splits(int64_t N, int64_t K, int rows_per_wg, int kc) {
  const int64_t blocks = (N + rows_per_wg - 1) / rows_per_wg;
  int S = 1;
  while (S < kStreamMaxSplits && blocks * 2 * S <= kStreamMaxWGs && K % (2ll * S * kc) == 0)
    S *= 2;
  return S;
}

// fp16 shapes whose unsplit 8-wave grid would leave many CUs idle (under
// kStreamMinWGs workgroups) take 6 waves per workgroup instead: more
// workgroups, each output summed by one wave in the same order as before
constexpr int kStreamNarrowKW = 6;
constexpr int64_t kStreamMinWGs = 192;

struct StreamPlan {
  bool fallback, narrow;
  int rows_per_wg, kc, splits;
};

template <bool W4, int MF>
static StreamPlan stream_plan_mf(int64_t N, int64_t K) {
  using P = StreamSel<W4, MF>;
  using B = StreamFallback<W4, MF>;
  StreamPlan pl;
  pl.fallback = K % P::KC != 0;
  pl.narrow = false;
  pl.rows_per_wg = pl.fallback ? 16 * B::NF * B::KW : 16 * P::NF * P::KW;
  pl.kc = pl.fallback ? B::KC : P::KC;
  pl.splits = stream_splits(N, K, pl.rows_per_wg, pl.kc);
  if (!W4 && !pl.fallback && pl.splits == 1) {
    const int rows6 = 16 * P::NF * kStreamNarrowKW;
    if ((N + pl.rows_per_wg - 1) / pl.rows_per_wg < kStreamMinWGs &&
        (N + rows6 - 1) / rows6 <= kStreamMaxWGs) {
      pl.narrow = true;
      pl.rows_per_wg = rows6;
    }
  }
  return pl;
}

static StreamPlan stream_plan(int64_t M, int64_t N, int64_t K, bool w4) {
  switch (stream_mf(M)) {
    case 2: return w4 ? stream_plan_mf<true, 2>(N, K) : stream_plan_mf<false, 2>(N, K);
    case 4: return w4 ? stream_plan_mf<true, 4>(N, K) : stream_plan_mf<false, 4>(N, K);
    default: return w4 ? stream_plan_mf<true, 8>(N, K) : stream_plan_mf<false, 8>(N, K);
  }
}

static bool uses_stream(int64_t M) { return M > 16 && M <= kStreamMaxM; }

int64_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, bool w4) {
  if (!uses_stream(M) || N <= 0 || K <= 0 || K % 128 != 0) return 0;
  const StreamPlan pl = stream_plan(M, N, K, w4);
  return pl.splits > 1 ? (int64_t)pl.splits * M * N * 4 : 0;
}

int64_t gemm_workspace_bytes_upto(int64_t M_max, int64_t N, int64_t K, bool w4) {
  int64_t best = 0;
  for (int64_t M : {(int64_t)32, (int64_t)64, (int64_t)kStreamMaxM}) {
    const int64_t m = M < M_max ? M : M_max;
    const int64_t b = gemm_workspace_bytes(m, N, K, w4);
    best = b > best ? b : best;
  }
  return best;
}

template <int NF, int MF, int KW, int PD, bool W4, int KC, int EPI, bool PK>
static void launch_stream_cfg(const GemmArgs& a, int S, float* ws, hipStream_t st) {
  constexpr int rows = 16 * NF * KW;
  const dim3 grid((unsigned)((a.N + rows - 1) / rows), (unsigned)S);
  launch((gemm_stream<NF, MF, KW, PD, W4, KC, EPI, PK>), grid, dim3(KW * 64), 0, st, a, ws,
         a.K / S);
  if (S > 1) launch_combine<EPI>(a, ws, S, st);
}

template <bool W4, int MF, int EPI, bool PK>
static void launch_stream_mf(const GemmArgs& a, const StreamPlan& pl, int S, float* ws,
                             hipStream_t st) {
  if (pl.fallback) {
    using B = StreamFallback<W4, MF>;
    launch_stream_cfg<B::NF, MF, B::KW, B::PD, W4, B::KC, EPI, PK>(a, S, ws, st);
  } else {
    using P = StreamSel<W4, MF>;
    if constexpr (!W4) {
      if (pl.narrow) {
        launch_stream_cfg<P::NF, MF, kStreamNarrowKW, P::PD, W4, P::KC, EPI, PK>(a, S, ws, st);
        return;
      }
    }
    launch_stream_cfg<P::NF, MF, P::KW, P::PD, W4, P::KC, EPI, PK>(a, S, ws, st);
  }
}

template <bool W4, int EPI, bool PK>
static pipo_status launch_epi(const GemmArgs& a, float* ws, int64_t ws_bytes, hipStream_t st) {
  if constexpr (EPI == EPI_SWIGLU) {
    (void)ws;
    (void)ws_bytes;
    if (a.M > 16) {
      set_error("gemm: the SwiGLU epilogue needs M <= 16 (M=%lld)", (long long)a.M);
      return PIPO_ERR_UNSUPPORTED;
    }
    launch_skinny<4, W4, EPI, PK>(a, st);
    PIPO_HIP_TRY(hipGetLastError());
    return PIPO_OK;
  } else {
    if (a.M <= 16) {
      // 64 W rows per workgroup (less X traffic per W byte) once that still
      // gives enough workgroups to fill the chip, else 16
      if (a.N >= 64 * 192)
        launch_skinny<4, W4, EPI, PK>(a, st);
      else
        launch_skinny<1, W4, EPI, PK>(a, st);
    } else if (a.M <= kStreamMaxM) {
      const StreamPlan pl = stream_plan(a.M, a.N, a.K, W4);
      // without room for the partial sums the K split is dropped
      const int S = (pl.splits > 1 && ws != nullptr && a.M * a.N < ((int64_t)1 << 31) &&
                     ws_bytes >= (int64_t)pl.splits * a.M * a.N * 4) ? pl.splits : 1;
      switch (stream_mf(a.M)) {
        case 2: launch_stream_mf<W4, 2, EPI, PK>(a, pl, S, ws, st); break;
        case 4: launch_stream_mf<W4, 4, EPI, PK>(a, pl, S, ws, st); break;
        default: launch_stream_mf<W4, 8, EPI, PK>(a, pl, S, ws, st); break;
      }
    } else if (big_tiles(a.M, a.N) >= kBigMinTiles) {
      const int64_t per_xcd = (big_tiles(a.M, a.N) + kXcds - 1) / kXcds;
      const dim3 grid((unsigned)(per_xcd * kXcds));
      if constexpr (W4)
        launch((gemm_big_w4<EPI, PK>), grid, dim3(kFThreads), 0, st, a);
      else
        launch((gemm_big_f16<EPI, PK>), grid, dim3(kFThreads), 0, st, a);
    } else {
      const int64_t total = ((a.N + kTBN - 1) / kTBN) * ((a.M + kTBM - 1) / kTBM);
      const int64_t per_xcd = (total + kXcds - 1) / kXcds;
      launch((gemm_tiled<W4, EPI, PK>), dim3((unsigned)(per_xcd * kXcds)), dim3(kTThreads), 0, st,
             a);
    }
    PIPO_HIP_TRY(hipGetLastError());
    return PIPO_OK;
  }
}

template <bool W4, bool PK>
static pipo_status launch_fmt(const GemmArgs& a, int epi, float* ws, int64_t ws_bytes,
                              hipStream_t st) {
  switch (epi) {
    case EPI_F16: return launch_epi<W4, EPI_F16, PK>(a, ws, ws_bytes, st);
    case EPI_RELU_F16: return launch_epi<W4, EPI_RELU_F16, PK>(a, ws, ws_bytes, st);
    case EPI_ADD_F32: return launch_epi<W4, EPI_ADD_F32, PK>(a, ws, ws_bytes, st);
    case EPI_F32: return launch_epi<W4, EPI_F32, PK>(a, ws, ws_bytes, st);
    case EPI_QKV: return launch_epi<W4, EPI_QKV, PK>(a, ws, ws_bytes, st);
    case EPI_SWIGLU: return launch_epi<W4, EPI_SWIGLU, PK>(a, ws, ws_bytes, st);
    default: set_error("gemm: unknown epilogue %d", epi); return PIPO_ERR_ARG;
  }
}

pipo_status launch_gemm(const GemmArgs& a, bool w4, int epi, float* workspace,
                        int64_t workspace_bytes, hipStream_t st) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) {
    set_error("gemm: empty shape M=%lld N=%lld K=%lld", (long long)a.M, (long long)a.N,
              (long long)a.K);
    return PIPO_ERR_ARG;
  }
  if (a.K % 128 != 0) {
    set_error("gemm: K=%lld is not a multiple of 128", (long long)a.K);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (a.X == nullptr || (w4 ? (a.Wq == nullptr || a.Wsm == nullptr) : a.W == nullptr)) {
    set_error("gemm: null operand");
    return PIPO_ERR_ARG;
  }
  if (a.M >= (int64_t(1) << 31)) {
    set_error("gemm: M=%lld rows exceeds 2^31 - 1", (long long)a.M);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (epi == EPI_QKV && a.rows_per_seq < 1) {
    set_error("gemm: QKV output with rows_per_seq=%lld", (long long)a.rows_per_seq);
    return PIPO_ERR_ARG;
  }
  if (epi == EPI_QKV && (a.dkv <= 0 || a.N != a.d + 2 * a.dkv)) {
    set_error("gemm: QKV output of %lld columns for d=%lld dkv=%lld", (long long)a.N,
              (long long)a.d, (long long)a.dkv);
    return PIPO_ERR_ARG;
  }
  if (epi == EPI_SWIGLU && (a.N % 2 != 0 || a.bias != nullptr || a.out16 == nullptr ||
                            a.ldo < a.N / 2)) {
    set_error("gemm: the SwiGLU epilogue needs an even N (gate over up rows), no bias and an "
              "fp16 output of N / 2 columns (N=%lld ldo=%lld)", (long long)a.N, (long long)a.ldo);
    return PIPO_ERR_ARG;
  }
  if (a.packed && a.N % 16 != 0) {
    set_error("gemm: fragment-ordered W needs N %% 16 == 0 (N=%lld)", (long long)a.N);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (a.packed)
    return w4 ? launch_fmt<true, true>(a, epi, workspace, workspace_bytes, st)
              : launch_fmt<false, true>(a, epi, workspace, workspace_bytes, st);
  return w4 ? launch_fmt<true, false>(a, epi, workspace, workspace_bytes, st)
            : launch_fmt<false, false>(a, epi, workspace, workspace_bytes, st);
}

}  // namespace pipo
