// Projection GEMMs of the decoder layer and the output head:
//   Y[M][N] = X[M][K] . W[N][K]^T  (+ bias, fused epilogue)
// with W in fp16 or group-wise INT4 (codes expanded to fp16 in registers,
// the paper's "compute directly on 4-bit weights", Section 3.4).
//
// Two kernels, chosen by M alone:
//   * gemm_skinny (M <= 64, decode): every workgroup owns 32 rows of W and
//     all M rows of X; its waves split K; W streams from HBM straight into
//     MFMA operand registers (no LDS), X comes from L2.  Partial sums are
//     combined across waves in LDS in a fixed order.
//   * gemm_tiled (M > 64, prefill): 128 x 128 output tiles, K staged through
//     double-buffered LDS in steps of 64, 4 waves of 64 x 64.
// Both accumulate in fp32 with v_mfma_f32_16x16x32_f16.  An output element
// depends only on its row of X, its row of W, K and the kernel choice, so
// launching a GEMM per chunk of W rows gives the same bits as one launch.
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
constexpr int kSkNF = 2;      // 16-row fragments of W per workgroup
constexpr int kSkWaves = 4;   // waves splitting K

template <int MF, bool W4, int EPI>
__global__ __launch_bounds__(kSkWaves * 64) void gemm_skinny(GemmArgs a) {
  constexpr int NF = kSkNF;
  __shared__ f4 red[kSkWaves][NF][MF][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * (16 * NF);
  const int64_t K = a.K;
  const int64_t nsteps = K / 128;

  f4 acc[NF][MF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) acc[f][mf] = f4{0.f, 0.f, 0.f, 0.f};

  // each lane owns 32 consecutive k of every 128-k step: kbase = 128 s + 32 g
  for (int64_t s = wave; s < nsteps; s += kSkWaves) {
    const int64_t kb = s * 128 + 32 * g;
    h8 wv[NF][4];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int64_t n = n0 + 16 * f + r;
      if (n < a.N) {
        if constexpr (W4) {
          const u32x4 codes = *reinterpret_cast<const u32x4*>(a.Wq + n * (K / 2) + kb / 2);
          const uint32_t smw = *reinterpret_cast<const uint32_t*>(a.Wsm + (n * (K / 64) + kb / 64) * 2);
          dequant32(codes, h2f((uint16_t)(smw & 0xFFFFu)), h2f((uint16_t)(smw >> 16)), wv[f]);
        } else {
          const uint16_t* p = a.W + n * K + kb;
#pragma unroll
          for (int i = 0; i < 4; ++i) wv[f][i] = load_h8(p + 8 * i);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) wv[f][i] = zero_h8();
      }
    }
    h8 xv[MF][4];
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) {
      const int64_t m = 16 * mf + r;
      if (m < a.M) {
        const uint16_t* p = a.X + m * K + kb;
#pragma unroll
        for (int i = 0; i < 4; ++i) xv[mf][i] = load_h8(p + 8 * i);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) xv[mf][i] = zero_h8();
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) acc[f][mf] = mfma16(wv[f][i], xv[mf][i], acc[f][mf]);
  }

#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) red[wave][f][mf][lane] = acc[f][mf];
  __syncthreads();

  // element (f, mf, lane', j): W row n0 + 16 f + 4 (lane' / 16) + j, X row 16 mf + lane' % 16
  constexpr int kElems = NF * MF * 64 * 4;
  for (int e = threadIdx.x; e < kElems; e += kSkWaves * 64) {
    const int j = e & 3;
    const int ln = (e >> 2) & 63;
    const int fm = e >> 8;
    const int f = fm / MF, mf = fm % MF;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kSkWaves; ++w) sum += red[w][f][mf][ln][j];
    const int64_t n = n0 + 16 * f + 4 * (ln >> 4) + j;
    const int64_t m = 16 * mf + (ln & 15);
    epilogue<EPI>(a, m, n, sum);
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
template <bool W4, int EPI>
static pipo_status launch_epi(const GemmArgs& a, hipStream_t st) {
  if (a.M <= 64) {
    const dim3 grid((unsigned)((a.N + 16 * kSkNF - 1) / (16 * kSkNF)));
    const dim3 block(kSkWaves * 64);
    const int mf = (int)((a.M + 15) / 16);
    switch (mf) {
      case 1: hipLaunchKernelGGL((gemm_skinny<1, W4, EPI>), grid, block, 0, st, a); break;
      case 2: hipLaunchKernelGGL((gemm_skinny<2, W4, EPI>), grid, block, 0, st, a); break;
      case 3: hipLaunchKernelGGL((gemm_skinny<3, W4, EPI>), grid, block, 0, st, a); break;
      default: hipLaunchKernelGGL((gemm_skinny<4, W4, EPI>), grid, block, 0, st, a); break;
    }
  } else {
    const dim3 grid((unsigned)((a.N + kTBN - 1) / kTBN), (unsigned)((a.M + kTBM - 1) / kTBM));
    hipLaunchKernelGGL((gemm_tiled<W4, EPI>), grid, dim3(kTThreads), 0, st, a);
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
