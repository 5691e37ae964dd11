// Shared host/device definitions of the pipelined-offloading decoder library.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <exception>
#include <functional>
#include <new>

#include "pipo.h"
#include "pipo_ops.h"

namespace pipo {

// thread-local error text behind pipo_last_error()
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

#define PIPO_HIP_TRY(call)                                                                  \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) {                                                                 \
      ::pipo::set_error("%s: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, __LINE__); \
      return PIPO_ERR_HIP;                                                                  \
    }                                                                                       \
  } while (0)

#define PIPO_TRY(expr)             \
  do {                             \
    pipo_status s_ = (expr);       \
    if (s_ != PIPO_OK) return s_;  \
  } while (0)

// Runs the body of a C entry point so that no C++ exception leaves it: an
// exhausted host heap (std::bad_alloc from a container or `new`) or any
// other exception of the host code becomes PIPO_ERR_OOM_HOST with its text.
template <typename F>
inline pipo_status guarded(F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    set_error("host memory allocation failed");
  } catch (const std::exception& e) {
    set_error("host resources exhausted: %s", e.what());
  } catch (...) {
    set_error("unexpected host exception");
  }
  return PIPO_ERR_OOM_HOST;
}

// fn(a, b) over the contiguous pieces of [0, n) cut into `nt` parts, each
// on a thread of its own; when the system refuses a thread, the caller runs
// the rest of the range itself, and every started thread is joined before
// the call returns.
void parallel_ranges(int64_t n, int64_t nt, const std::function<void(int64_t, int64_t)>& fn);

// Events that bracket the kernel launches of one operation made on this
// thread.  They are attached to the dispatches themselves
// (hipExtLaunchKernelGGL), so they time the kernels rather than the
// stream's progress around them: `start` marks the start of the first
// dispatch, and `stop` is re-recorded at the end of every dispatch until the
// caller clears it, so an operation of several kernels (a split GEMM and its
// combine) is timed from its first kernel's start to its last one's end.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& next_launch_events();

template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t st, Args... args) {
  LaunchEvents& ev = next_launch_events();
  if (ev.start || ev.stop) {
    const LaunchEvents e = ev;
    ev.start = nullptr;
    hipExtLaunchKernelGGL(kernel, grid, block, lds, st, e.start, e.stop, 0u, args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, lds, st, args...);
  }
}

// GEMM epilogues (the first four are the public PIPO_EPI_* values)
enum : int {
  EPI_F16 = PIPO_EPI_F16,
  EPI_RELU_F16 = PIPO_EPI_RELU_F16,
  EPI_ADD_F32 = PIPO_EPI_ADD_F32,
  EPI_F32 = PIPO_EPI_F32,
  EPI_QKV = 4,  // q (scaled) to q_out, k and v rows into a position-major KV cache
  EPI_SWIGLU = PIPO_EPI_SWIGLU,  // gate and up rows stacked in W; silu(g) * u to out16
};

struct GemmArgs {
  const uint16_t* X = nullptr;    // [M][K] fp16
  const uint16_t* W = nullptr;    // [N][K] fp16
  const uint8_t* Wq = nullptr;    // [N][K/2] int4 codes
  const uint16_t* Wsm = nullptr;  // [N][K/64][2] fp16 (scale, min)
  const uint16_t* bias = nullptr; // [N] fp16 or null
  int64_t M = 0, N = 0, K = 0;
  bool packed = false;            // W (or Wq, Wsm) in fragment order (device.h)
  uint16_t* out16 = nullptr;      // [M][ldo]
  float* out32 = nullptr;         // [M][ldo]
  int64_t ldo = 0;
  // EPI_QKV: row m is sequence m / rows_per_seq at position pos0 + m % rows_per_seq;
  // output columns [0, d) are q, the next dkv k, the last dkv v (dkv = d
  // without grouped-query attention)
  uint16_t* q_out = nullptr;      // [M][d]
  uint16_t* k_out = nullptr;      // cache rows (p * batch + seq), [.][dkv]
  uint16_t* v_out = nullptr;
  int64_t d = 0, dkv = 0;
  float q_scale = 1.f;
  int64_t rows_per_seq = 1, pos0 = 0, batch = 1;
};

// kernel launchers (gemm.hip, attention.hip, elementwise.hip)
// 16 < M <= 128 may split K over workgroups; their partial sums need
// `workspace` (gemm_workspace_bytes; contents arbitrary, not shared by
// overlapping launches).  With less the GEMM runs unsplit, equal up to
// rounding.  gemm_workspace_bytes_upto covers every M up to M_max.
pipo_status launch_gemm(const GemmArgs& a, bool w4, int epi, float* workspace,
                        int64_t workspace_bytes, hipStream_t st);
int64_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, bool w4);
int64_t gemm_workspace_bytes_upto(int64_t M_max, int64_t N, int64_t K, bool w4);
pipo_status launch_layernorm(const float* x, const uint16_t* g, const uint16_t* b, uint16_t* y,
                             int64_t rows, int64_t d, int64_t src_stride, int64_t src_offset,
                             float eps, hipStream_t st);
// y = x / sqrt(mean(x^2) + eps) * g (RMSNorm), same row addressing as LayerNorm
pipo_status launch_rmsnorm(const float* x, const uint16_t* g, uint16_t* y, int64_t rows,
                           int64_t d, int64_t src_stride, int64_t src_offset, float eps,
                           hipStream_t st);
// pos_table may be null (no learned positions)
pipo_status launch_embed(const uint16_t* tok_rows, const int32_t* ids, const uint16_t* tok_table,
                         const uint16_t* pos_table, float* x, int64_t rows, int64_t d,
                         int64_t rows_per_seq, int64_t pos0, int64_t pos_offset, hipStream_t st);
// rotary positions, in place: q rows [M][H * D] (then scaled by q_scale) and
// k rows at cache row (kpos0 + m % rows_per_seq) * batch + m / rows_per_seq of
// [.][Hkv * D]; row m sits at position pos0 + m % rows_per_seq, whose
// (cos, sin) pairs are cs[pos][D / 2][2]
pipo_status launch_rope(uint16_t* q, uint16_t* k, const float* cs, int64_t M,
                        int64_t rows_per_seq, int64_t pos0, int64_t kpos0, int64_t batch, int H,
                        int Hkv, int D, float q_scale, hipStream_t st);
// h[m][i] = silu(gu[m][i]) * gu[m][F + i]
pipo_status launch_swiglu(const uint16_t* gu, uint16_t* h, int64_t M, int64_t F, hipStream_t st);
// decode attention splits the keys of a (sequence, head) over several
// workgroups when there are few of them; the splits' partial results go to
// `workspace` (attn_decode_workspace_bytes) and a second kernel merges them
// in split order; without enough workspace it runs unsplit
// Query head h reads key/value head h / (n_heads / n_kv_heads); cache rows
// hold the n_kv_heads heads side by side.
// heads of a decode-attention workgroup: 4, 2 or 1 adjacent heads without
// grouping, one key/value head (and its query heads) with it; kv4: INT4 rows
int attn_decode_heads_per_wg(int b, int n_heads, int n_kv_heads, bool kv4);
int attn_decode_splits(int b, int n_heads, int n_kv_heads, int t, bool kv4);
int64_t attn_decode_workspace_bytes(int b, int n_heads, int head_dim, int splits);
// kc, vc: fp16 rows, or INT4 rows (kv4; see kvcache.hip) of the cache
pipo_status launch_attn_decode(const uint16_t* q, const void* kc, const void* vc, uint16_t* o,
                               int b, int n_heads, int n_kv_heads, int head_dim, int t, bool kv4,
                               float* workspace, int64_t workspace_bytes, hipStream_t st);
pipo_status launch_attn_prefill(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                uint16_t* o, int b, int P, int n_heads, int n_kv_heads,
                                int head_dim, hipStream_t st);
// INT4 KV rows (d/2 code bytes + d/64 fp16 (scale, min) pairs; d % 256 == 0)
pipo_status launch_kv_quant(const uint16_t* x, uint8_t* out, int64_t rows, int64_t d,
                            hipStream_t st);
pipo_status launch_kv_dequant(const uint8_t* in, uint16_t* y, int64_t rows, int64_t d,
                              hipStream_t st);
// greedy argmax (largest, ties to the lowest index, NaNs skipped); with a
// workspace of argmax_workspace_bytes a row is split over several
// workgroups and a second kernel merges their candidates (same result)
int64_t argmax_workspace_bytes(int64_t rows, int64_t V);
pipo_status launch_argmax(const float* logits, int32_t* next, int64_t rows, int64_t V,
                          void* workspace, int64_t workspace_bytes, hipStream_t st);
pipo_status launch_fill_u16(uint16_t* p, uint16_t value, int64_t n, hipStream_t st);
pipo_status launch_copy16(void* dst, const void* src, int64_t bytes, hipStream_t st);

// longest context the decode-attention path accepts, and its split cap
constexpr int kAttnDecodeMaxT = 65536;
constexpr int kAttnDecodeMaxSplits = 16;
constexpr int kAttnDecodeMinWGs = 768;
constexpr int kAttnDecodeWideWGs = 1536;

}  // namespace pipo
