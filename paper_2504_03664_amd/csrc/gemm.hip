// Projection GEMMs of the decoder layer and the output head:
//   Y[M][N] = X[M][K] . W[N][K]^T  (+ bias, fused epilogue)
// with W in fp16 or group-wise INT4 (codes expanded to fp16 in registers,
// the paper's "compute directly on 4-bit weights", Section 3.4).
//
// Two kernels, chosen by M alone:
//   * gemm_skinny (M <= 64, decode): every workgroup owns 16 or 64 rows of
//     W and all M rows of X; its waves split K; W streams from HBM straight
//     into MFMA operand registers (no LDS), X comes from L2.  Partial sums
//     are combined across waves in LDS in a fixed order.
//   * gemm_tiled (M > 64, prefill): 128 x 128 output tiles, K staged through
//     double-buffered LDS in steps of 64, 4 waves of 64 x 64.
// Both accumulate in fp32 with v_mfma_f32_16x16x32_f16.  The summation order
// of an element depends only on M (kernel and waves) and K, so a launch over
// any row range of W gives the same bits for those rows as a full launch,
// and no workgroup ever reads another workgroup's results.
#include "common.h"
#include "device.h"

namespace pipo {

template <int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int64_t m, int64_t n, float acc) {
  if (m >= a.M || n >= a.N) return;
  const float v = acc + (a.bias ? h2f(a.bias[n]) : 0.f);
  if constexpr (EPI == EPI_F16) {
    a.out16[m * a.ldo + n] = f2h(v);
  } else if constexpr (EPI == EPI_RELU_F16) {
    a.out16[m * a.ldo + n] = f2h(v > 0.f ? v : 0.f);
  } else if constexpr (EPI == EPI_ADD_F32) {
    a.out32[m * a.ldo + n] += v;
  } else if constexpr (EPI == EPI_F32) {
    a.out32[m * a.ldo + n] = v;
  } else {  // EPI_QKV
    const int64_t seq = m / a.rows_per_seq;
    const int64_t pos = a.pos0 + m % a.rows_per_seq;
    const int64_t crow = pos * a.batch + seq;
    if (n < a.d) {
      a.q_out[m * a.d + n] = f2h(v * a.q_scale);
    } else if (n < 2 * a.d) {
      a.k_out[crow * a.d + (n - a.d)] = f2h(v);
    } else {
      a.v_out[crow * a.d + (n - 2 * a.d)] = f2h(v);
    }
  }
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
template <int NF, int MF, int KW, int UNR, bool W4>
struct SkinnyStep {
  u32x4 w[NF][4];  // fp16: four 8-half chunks; int4: w[f][0] holds 32 codes
  uint32_t sm[NF];
  h8 x[MF][4];

  __device__ __forceinline__ static int koff(int i, int g) { return W4 ? 32 * g + 8 * i : 32 * i + 8 * g; }

  __device__ __forceinline__ void load(const GemmArgs& a, int64_t n0, int64_t s, int r, int g) {
    const int64_t K = a.K;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int64_t n = n0 + 16 * f + r;
      const bool ok = n < a.N;
      if constexpr (W4) {
        const int64_t kb = s * 128 + 32 * g;
        w[f][0] = ok ? *reinterpret_cast<const u32x4*>(a.Wq + n * (K / 2) + kb / 2)
                     : u32x4{0, 0, 0, 0};
        sm[f] = ok ? *reinterpret_cast<const uint32_t*>(a.Wsm + (n * (K / 64) + kb / 64) * 2) : 0u;
      } else {
        const uint16_t* p = a.W + n * K + s * 128;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          w[f][i] = ok ? *reinterpret_cast<const u32x4*>(p + koff(i, g)) : u32x4{0, 0, 0, 0};
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
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      h8 wv[4];
      if constexpr (W4) {
        dequant32(w[f][0], h2f((uint16_t)(sm[f] & 0xFFFFu)), h2f((uint16_t)(sm[f] >> 16)), wv);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) wv[i] = __builtin_bit_cast(h8, w[f][i]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) acc[f][mf] = mfma16(wv[i], x[mf][i], acc[f][mf]);
    }
  }
};

template <int NF, int MF, int KW, int UNR, bool W4, int EPI>
__global__ __launch_bounds__(KW * 64) void gemm_skinny(GemmArgs a) {
  __shared__ f4 red[KW][NF][MF][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * (16 * NF);
  const int64_t nsteps = a.K / 128;

  f4 acc[NF][MF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) acc[f][mf] = f4{0.f, 0.f, 0.f, 0.f};

  for (int64_t s = wave; s < nsteps; s += UNR * KW) {
    SkinnyStep<NF, MF, KW, UNR, W4> st[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (s + u * KW < nsteps) st[u].load(a, n0, s + u * KW, r, g);
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (s + u * KW < nsteps) st[u].mma(acc);
  }

#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) red[wave][f][mf][lane] = acc[f][mf];
  __syncthreads();

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

// ---------------------------------------------------------------------------
// tiled GEMM (prefill)
constexpr int kTBM = 128, kTBN = 128, kTBK = 64, kTPad = 8;
constexpr int kTThreads = 256;  // 2 x 2 waves of 64 x 64

template <bool W4, int EPI>
__global__ __launch_bounds__(kTThreads) void gemm_tiled(GemmArgs a) {
  constexpr int LDS_ROW = kTBK + kTPad;  // halves
  __shared__ __attribute__((aligned(16))) uint16_t As[2][kTBM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][kTBN * LDS_ROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.y * kTBM;
  const int64_t n0 = (int64_t)blockIdx.x * kTBN;
  const int64_t K = a.K;
  const int64_t KT = K / kTBK;

  // global -> register staging: A and fp16 B take 4 chunks of 8 halves per
  // thread (row = c / 8, col = 8 (c % 8)); INT4 B takes one 32-code chunk.
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
      const int row = tid >> 1, half = tid & 1;
      const int64_t n = n0 + row;
      if (n < a.N) {
        const u32x4 codes =
            *reinterpret_cast<const u32x4*>(a.Wq + n * (K / 2) + kt * (kTBK / 2) + half * 16);
        const uint32_t smw = *reinterpret_cast<const uint32_t*>(a.Wsm + (n * (K / 64) + kt) * 2);
        dequant32(codes, h2f((uint16_t)(smw & 0xFFFFu)), h2f((uint16_t)(smw >> 16)), rb);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) rb[i] = zero_h8();
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + i * kTThreads;
        const int row = c >> 3, col = (c & 7) * 8;
        const int64_t n = n0 + row;
        rb[i] = n < a.N ? load_h8(a.W + n * K + kt * kTBK + col) : zero_h8();
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
      const int row = tid >> 1, half = tid & 1;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<h8*>(&Bs[buf][row * LDS_ROW + half * 32 + 8 * i]) = rb[i];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + i * kTThreads;
        const int row = c >> 3, col = (c & 7) * 8;
        *reinterpret_cast<h8*>(&Bs[buf][row * LDS_ROW + col]) = rb[i];
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

  // acc[i][j] element e: row m0 + 64 wm + 16 i + 4 g + e, col n0 + 64 wn + 16 j + r
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        epilogue<EPI>(a, m0 + wm * 64 + i * 16 + 4 * g + e, n0 + wn * 64 + j * 16 + r,
                      acc[i][j][e]);
}

// ---------------------------------------------------------------------------
// skinny configurations by M: (waves, steps in flight per wave)
template <int MF> struct SkinnyCfg;
template <> struct SkinnyCfg<1> { static constexpr int KW = 8, UNR = 2; };
template <> struct SkinnyCfg<2> { static constexpr int KW = 8, UNR = 1; };
template <> struct SkinnyCfg<4> { static constexpr int KW = 4, UNR = 1; };

template <int NF, int MF, bool W4, int EPI>
static void launch_skinny(const GemmArgs& a, hipStream_t st) {
  using C = SkinnyCfg<MF>;
  const dim3 grid((unsigned)((a.N + 16 * NF - 1) / (16 * NF)));
  launch((gemm_skinny<NF, MF, C::KW, C::UNR, W4, EPI>), grid, dim3(C::KW * 64), 0, st, a);
}

template <int NF, bool W4, int EPI>
static void launch_skinny_m(const GemmArgs& a, hipStream_t st) {
  if (a.M <= 16)
    launch_skinny<NF, 1, W4, EPI>(a, st);
  else if (a.M <= 32)
    launch_skinny<NF, 2, W4, EPI>(a, st);
  else
    launch_skinny<NF, 4, W4, EPI>(a, st);
}

template <bool W4, int EPI>
static pipo_status launch_epi(const GemmArgs& a, hipStream_t st) {
  if (a.M <= 64) {
    // 64 W rows per workgroup (less X traffic per W byte) once that still
    // gives enough workgroups to fill the chip, else 16
    if (a.N >= 64 * 192)
      launch_skinny_m<4, W4, EPI>(a, st);
    else
      launch_skinny_m<1, W4, EPI>(a, st);
  } else {
    const dim3 grid((unsigned)((a.N + kTBN - 1) / kTBN), (unsigned)((a.M + kTBM - 1) / kTBM));
    launch((gemm_tiled<W4, EPI>), grid, dim3(kTThreads), 0, st, a);
  }
  PIPO_HIP_TRY(hipGetLastError());
  return PIPO_OK;
}

template <bool W4>
static pipo_status launch_fmt(const GemmArgs& a, int epi, hipStream_t st) {
  switch (epi) {
    case EPI_F16: return launch_epi<W4, EPI_F16>(a, st);
    case EPI_RELU_F16: return launch_epi<W4, EPI_RELU_F16>(a, st);
    case EPI_ADD_F32: return launch_epi<W4, EPI_ADD_F32>(a, st);
    case EPI_F32: return launch_epi<W4, EPI_F32>(a, st);
    case EPI_QKV: return launch_epi<W4, EPI_QKV>(a, st);
    default: set_error("gemm: unknown epilogue %d", epi); return PIPO_ERR_ARG;
  }
}

pipo_status launch_gemm(const GemmArgs& a, bool w4, int epi, hipStream_t st) {
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
  return w4 ? launch_fmt<true>(a, epi, st) : launch_fmt<false>(a, epi, st);
}

}  // namespace pipo
