/*
 * pipo_ops.h -- the decoder's individual GPU operations, exposed for unit
 * tests and profiling.  Each call enqueues one operation of the layer
 * computation (PIPO's "Computation" task, Section 3.1.2) on `stream`
 * (a hipStream_t, or NULL for the default stream) and returns without
 * waiting.  All tensor pointers are device pointers unless stated;
 * ownership stays with the caller.  Shapes outside a kernel's range return
 * PIPO_ERR_UNSUPPORTED before anything is launched.
 */
#ifndef PIPO_OPS_H
#define PIPO_OPS_H

#include "pipo.h"

#ifdef __cplusplus
extern "C" {
#endif

/* --- device memory helpers (so tests need no other GPU runtime) --- */
pipo_status pipo_dev_alloc(size_t bytes, void** out);
pipo_status pipo_dev_free(void* p);
pipo_status pipo_copy_h2d(void* dst_dev, const void* src_host, size_t bytes);
pipo_status pipo_copy_d2h(void* dst_host, const void* src_dev, size_t bytes);
pipo_status pipo_dev_synchronize(void);

/* GEMM epilogues: acc = X[m] . W[n] (fp32), then
 *   PIPO_EPI_F16:       out_f16[m][n] = acc + bias[n]
 *   PIPO_EPI_RELU_F16:  out_f16[m][n] = max(acc + bias[n], 0)
 *   PIPO_EPI_ADD_F32:   out_f32[m][n] += acc + bias[n]     (residual stream)
 *   PIPO_EPI_F32:       out_f32[m][n] = acc + bias[n]      (logits)
 * bias may be NULL (treated as 0). */
enum { PIPO_EPI_F16 = 0, PIPO_EPI_RELU_F16 = 1, PIPO_EPI_ADD_F32 = 2, PIPO_EPI_F32 = 3 };

/*
 * Y = X . W^T with the chosen epilogue (the projections of a layer and the
 * output head).  X: [M][K] fp16 (row stride K); W: [N][K] fp16; out: [M][N]
 * (row stride N), fp16 or fp32 per epilogue.  K must be a multiple of 128.
 * For 16 < M <= 128 the K range may be split over workgroups whose fp32
 * partial sums go to `workspace` (device, caller-owned, contents
 * arbitrary) of pipo_op_gemm_workspace_bytes(M, N, K, wfmt) bytes; a second
 * kernel adds them in a fixed order and applies the epilogue.  With less
 * (or NULL) workspace the GEMM runs unsplit; the result is the same up to
 * rounding.  Calls sharing a workspace must not overlap in time.  For a
 * given (M, N, K, workspace sufficient or not) the summation order is
 * fixed, so repeated calls give the same bits.
 */
pipo_status pipo_op_gemm_f16(const uint16_t* X, const uint16_t* W, const uint16_t* bias,
                             void* out, int64_t M, int64_t N, int64_t K, int32_t epi,
                             void* workspace, int64_t workspace_bytes, void* stream);

/* Same with group-wise INT4 W (pipo_q4 layout, device pointers): the codes
 * are expanded to fp16 inside the GEMM (Section 3.4), never in HBM; every
 * code becomes code * scale + min rounded once to fp16. */
pipo_status pipo_op_gemm_w4(const uint16_t* X, const uint8_t* Wq, const uint16_t* Wsm,
                            const uint16_t* bias, void* out, int64_t M, int64_t N, int64_t K,
                            int32_t epi, void* workspace, int64_t workspace_bytes,
                            void* stream);

/* Workspace bytes the GEMM of this shape uses to split K (0: never splits).
 * wfmt: PIPO_W_FP16 or PIPO_W_INT4_G64. */
int64_t pipo_op_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int32_t wfmt);

/* y[r][:] = LN(x[r*src_stride + src_offset][:]) * gamma + beta, r < rows;
 * x fp32 [.][d], y fp16 [rows][d], statistics in fp32. */
pipo_status pipo_op_layernorm(const float* x, const uint16_t* gamma, const uint16_t* beta,
                              uint16_t* y, int64_t rows, int64_t d, int64_t src_stride,
                              int64_t src_offset, float eps, void* stream);

/*
 * Decode attention for b sequences at position t (keys 0..t visible).
 * q: [b][d] fp16 (already scaled by head_dim^-1/2); kc, vc: KV cache
 * [>= t+1][b][d] fp16 (position-major: row p*b + i holds sequence i's key at
 * position p); o: [b][d] fp16.  head_dim 64 or 128, t + 1 <= 65536.
 * When b * n_heads is small the keys are split over several workgroups and
 * a second kernel merges the splits in order; the partials need `workspace`
 * (device, caller-owned, contents arbitrary) of
 * pipo_op_attn_decode_workspace_bytes(b, n_heads, head_dim, t) bytes.  With
 * less (or NULL) the kernel runs unsplit; the result is the same up to
 * rounding.  Calls sharing a workspace must not overlap in time.
 */
pipo_status pipo_op_attn_decode(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                uint16_t* o, int32_t b, int32_t n_heads, int32_t head_dim,
                                int32_t t, void* workspace, int64_t workspace_bytes,
                                void* stream);
int64_t pipo_op_attn_decode_workspace_bytes(int32_t b, int32_t n_heads, int32_t head_dim,
                                            int32_t t);

/* The same over an INT4 KV cache (PIPO_KV_INT4_G64 rows of 9d/16 bytes,
 * position-major like the fp16 cache; d % 256 == 0): every key and value
 * is read as code * scale + min (rounded once to fp16).  Same workspace. */
pipo_status pipo_op_attn_decode_kv4(const uint16_t* q, const uint8_t* kc, const uint8_t* vc,
                                    uint16_t* o, int32_t b, int32_t n_heads, int32_t head_dim,
                                    int32_t t, void* workspace, int64_t workspace_bytes,
                                    void* stream);

/* INT4 KV cache rows (Section 2; the conversion is part of saving and
 * loading the cache, Section 3.1.2): quantize `rows` fp16 rows x [rows][d]
 * into out [rows][9d/16 bytes] with the PIPO_KV_INT4_G64 recipe (pipo.h),
 * or expand INT4 rows back to fp16 y [rows][d].  d % 256 == 0. */
pipo_status pipo_op_kv_quant(const uint16_t* x, uint8_t* out, int64_t rows, int64_t d,
                             void* stream);
pipo_status pipo_op_kv_dequant(const uint8_t* in, uint16_t* y, int64_t rows, int64_t d,
                               void* stream);

/*
 * Causal prefill attention over P positions of b sequences.
 * q: [b][P][d] fp16 (scaled); kc, vc: [>= P][b][d] position-major as
 * above; o: [b][P][d] fp16.  head_dim 64 or 128.
 */
pipo_status pipo_op_attn_prefill(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                 uint16_t* o, int32_t b, int32_t P, int32_t n_heads,
                                 int32_t head_dim, void* stream);

/* next[r] = index of the largest logits[r][:] (ties: lowest index). */
pipo_status pipo_op_argmax(const float* logits, int32_t* next, int64_t rows, int64_t V,
                           void* stream);

/* Plain device-to-device copy kernel: reads and writes `bytes` once
 * (multiple of 16, 16-byte aligned pointers).  Not part of the decoder: it
 * gives a kernel of known HBM traffic for calibrating hardware counters. */
pipo_status pipo_op_copy(void* dst, const void* src, int64_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PIPO_OPS_H */
