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
 * bias may be NULL (treated as 0).
 *   PIPO_EPI_SWIGLU:    the gated MLP's SwiGLU (LLaMA): W stacks the gate rows
 *                       [0, F) over the up rows [F, 2F) (N = 2F, even), bias
 *                       must be NULL, out_f16 has F columns (row stride F):
 *                       out_f16[m][i] = silu(g) * u in fp32, rounded once, with
 *                       g = fp16(acc of row i), u = fp16(acc of row F + i),
 *                       silu(g) = g / (1 + exp(-g)); the same values as
 *                       PIPO_EPI_F16 followed by pipo_op_swiglu.  Only for
 *                       M <= 16 (else PIPO_ERR_UNSUPPORTED). */
enum { PIPO_EPI_F16 = 0, PIPO_EPI_RELU_F16 = 1, PIPO_EPI_ADD_F32 = 2, PIPO_EPI_F32 = 3,
       PIPO_EPI_SWIGLU = 5 };

/*
 * Y = X . W^T with the chosen epilogue (the projections of a layer and the
 * output head).  X: [M][K] fp16 (row stride K); W: [N][K] fp16; out: [M][N]
 * (row stride N), fp16 or fp32 per epilogue ([M][N/2] fp16 for
 * PIPO_EPI_SWIGLU).  K must be a multiple of 128 and M below 2^31 (else
 * PIPO_ERR_UNSUPPORTED).
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

/* The same two GEMMs with W (or Wq, Wsm) in PIPO_LAYOUT_FRAGMENT order
 * (pipo.h; N % 16 == 0): same kernels, same summation order, so the result
 * equals the row-major call bit for bit. */
pipo_status pipo_op_gemm_f16_frag(const uint16_t* X, const uint16_t* W, const uint16_t* bias,
                                  void* out, int64_t M, int64_t N, int64_t K, int32_t epi,
                                  void* workspace, int64_t workspace_bytes, void* stream);
pipo_status pipo_op_gemm_w4_frag(const uint16_t* X, const uint8_t* Wq, const uint16_t* Wsm,
                                 const uint16_t* bias, void* out, int64_t M, int64_t N,
                                 int64_t K, int32_t epi, void* workspace,
                                 int64_t workspace_bytes, void* stream);

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
 * position p); o: [b][d] fp16.  head_dim 64 or 128, t + 1 <= 65536 (beyond:
 * PIPO_ERR_UNSUPPORTED).
 * When b * n_heads is small the keys are split over several workgroups and
 * a second kernel merges the splits in order; the partials need `workspace`
 * (device, caller-owned, contents arbitrary) of
 * pipo_op_attn_decode_workspace_bytes(b, n_heads, head_dim, t) bytes.  With
 * less (or NULL) the kernel runs unsplit; the result is the same up to
 * rounding.  Calls sharing a workspace must not overlap in time.  The
 * workspace size covers this call and pipo_op_attn_decode_kv4 alike.
 */
pipo_status pipo_op_attn_decode(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                uint16_t* o, int32_t b, int32_t n_heads, int32_t head_dim,
                                int32_t t, void* workspace, int64_t workspace_bytes,
                                void* stream);
int64_t pipo_op_attn_decode_workspace_bytes(int32_t b, int32_t n_heads, int32_t head_dim,
                                            int32_t t);

/*
 * pipo_op_attn_decode for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid
 * hipMalloc): the same kernels, split choice and result bit for bit as
 * pipo_op_attn_decode with a sufficient workspace, but the split partials
 * go to one fixed 4 MiB array of the library on each device (held until
 * the process ends) instead of a caller workspace; nothing is allocated.
 * Every shape this kernel accepts needs at most about 0.8 MB of it; a
 * shape that would need more returns PIPO_ERR_UNSUPPORTED.  All calls on a
 * device share that array, so calls that overlap in time on one device
 * (on different streams, or from several threads) race and must be
 * serialised by the caller.  The array's contents are arbitrary between
 * calls (every partial is written before it is read).
 */
pipo_status pipo_op_attn_decode_noalloc(const uint16_t* q, const uint16_t* kc,
                                        const uint16_t* vc, uint16_t* o, int32_t b,
                                        int32_t n_heads, int32_t head_dim, int32_t t,
                                        void* stream);

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
 * above; o: [b][P][d] fp16.  head_dim 64 or 128.  b * d * 64 (64 cached
 * positions of every sequence) must stay below 2^31 elements, else
 * PIPO_ERR_UNSUPPORTED.
 */
pipo_status pipo_op_attn_prefill(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                 uint16_t* o, int32_t b, int32_t P, int32_t n_heads,
                                 int32_t head_dim, void* stream);

/* --- LLaMA-family operations (PIPO_FAMILY_LLAMA in pipo.h) --- */

/* Grouped-query decode attention: q [b][n_heads * head_dim], cache rows of
 * n_kv_heads * head_dim (fp16, or PIPO_KV_INT4_G64 rows when kv_fmt says
 * so, then n_kv_heads * head_dim % 256 == 0); query head h reads key/value
 * head h / (n_heads / n_kv_heads), 1, 2, 4 or 8 query heads per key/value
 * head.  One workgroup serves all query heads of a key/value head, so each
 * cached row is read once.  Workspace as for pipo_op_attn_decode, sized by
 * pipo_op_attn_decode_gqa_workspace_bytes. */
pipo_status pipo_op_attn_decode_gqa(const uint16_t* q, const void* kc, const void* vc,
                                    uint16_t* o, int32_t b, int32_t n_heads, int32_t n_kv_heads,
                                    int32_t head_dim, int32_t t, int32_t kv_fmt, void* workspace,
                                    int64_t workspace_bytes, void* stream);
int64_t pipo_op_attn_decode_gqa_workspace_bytes(int32_t b, int32_t n_heads, int32_t n_kv_heads,
                                                int32_t head_dim, int32_t t);

/* Grouped-query causal prefill attention (layouts as pipo_op_attn_prefill,
 * cache rows of n_kv_heads * head_dim). */
pipo_status pipo_op_attn_prefill_gqa(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                     uint16_t* o, int32_t b, int32_t P, int32_t n_heads,
                                     int32_t n_kv_heads, int32_t head_dim, void* stream);

/* RMSNorm: y[r][:] = x[src] / sqrt(mean(x[src]^2) + eps) * gamma with
 * src = r*src_stride + src_offset; x fp32, y fp16, statistics in fp32. */
pipo_status pipo_op_rmsnorm(const float* x, const uint16_t* gamma, uint16_t* y, int64_t rows,
                            int64_t d, int64_t src_stride, int64_t src_offset, float eps,
                            void* stream);

/*
 * Rotary positions, in place (pipo.h, PIPO_FAMILY_LLAMA).  Row m (m < M)
 * is sequence m / rows_per_seq at position pos0 + m % rows_per_seq.
 * q: [M][n_heads * head_dim] fp16, each head rotated and then multiplied by
 * q_scale; k: rows (kpos0 + m % rows_per_seq) * batch + m / rows_per_seq of
 * [.][n_kv_heads * head_dim] fp16 (a position-major cache, or with kpos0 = 0
 * a staging buffer), rotated.  cos_sin: device fp32 [positions][head_dim/2]
 * [2] = (cos, sin) of p * w_i (pipo_rope_table).  head_dim 64 or 128.
 */
pipo_status pipo_op_rope(uint16_t* q, uint16_t* k, const float* cos_sin, int64_t M,
                         int64_t rows_per_seq, int64_t pos0, int64_t kpos0, int64_t batch,
                         int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, float q_scale,
                         void* stream);

/* The rotary table of a LLaMA shape on the host: out[p][i][2] = (cos, sin)
 * of p * w_i (w_i as in pipo.h, with the 3.1 scaling when rope_factor >
 * 0), computed in double and stored as fp32, for p < n_pos and i <
 * head_dim / 2.  `out` holds n_pos * head_dim floats.  Errors: ARG. */
pipo_status pipo_rope_table(const pipo_shape* shape, int32_t n_pos, float* out);

/* SwiGLU: h[m][i] = silu(gu[m][i]) * gu[m][F + i], silu(g) = g / (1 +
 * exp(-g)), in fp32; gu [M][2F], h [M][F] fp16, F % 8 == 0. */
pipo_status pipo_op_swiglu(const uint16_t* gu, uint16_t* h, int64_t M, int64_t F, void* stream);

/* Embedding: x[r][:] = tok_table[ids[r]] (+ pos_table[pos0 + r % rows_per_seq
 * + pos_offset] when pos_table is not NULL), fp32 x [rows][d]. */
pipo_status pipo_op_embed(const int32_t* ids, const uint16_t* tok_table, const uint16_t* pos_table,
                          float* x, int64_t rows, int64_t d, int64_t rows_per_seq, int64_t pos0,
                          int64_t pos_offset, void* stream);

/* next[r] = index of the largest logits[r][:] (ties: lowest index, NaNs
 * skipped; a row of NaNs gives 0).  rows <= 65535. */
pipo_status pipo_op_argmax(const float* logits, int32_t* next, int64_t rows, int64_t V,
                           void* stream);
/* The same with a row split over several workgroups whose candidates a
 * second kernel merges (same result); workspace (device, caller-owned,
 * contents arbitrary) of pipo_op_argmax_workspace_bytes(rows, V) bytes, or
 * less / NULL for the single-pass kernel. */
pipo_status pipo_op_argmax_ws(const float* logits, int32_t* next, int64_t rows, int64_t V,
                              void* workspace, int64_t workspace_bytes, void* stream);
int64_t pipo_op_argmax_workspace_bytes(int64_t rows, int64_t V);

/* Plain device-to-device copy kernel: reads and writes `bytes` once
 * (multiple of 16, 16-byte aligned pointers).  Not part of the decoder: it
 * gives a kernel of known HBM traffic for calibrating hardware counters. */
pipo_status pipo_op_copy(void* dst, const void* src, int64_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PIPO_OPS_H */
