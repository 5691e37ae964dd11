// C ABI of the individual operations (include/pipo_ops.h).
#include "common.h"

using namespace pipo;

extern "C" {

pipo_status pipo_dev_alloc(size_t bytes, void** out) {
  clear_error();
  if (!out) {
    set_error("out is NULL");
    return PIPO_ERR_ARG;
  }
  *out = nullptr;
  if (bytes == 0) return PIPO_OK;
  if (hipMalloc(out, bytes) != hipSuccess) {
    (void)hipGetLastError();
    *out = nullptr;
    set_error("hipMalloc of %zu bytes failed", bytes);
    return PIPO_ERR_OOM_DEVICE;
  }
  return PIPO_OK;
}

pipo_status pipo_dev_free(void* p) {
  clear_error();
  if (p) PIPO_HIP_TRY(hipFree(p));
  return PIPO_OK;
}

pipo_status pipo_copy_h2d(void* dst, const void* src, size_t bytes) {
  clear_error();
  if (bytes) PIPO_HIP_TRY(hipMemcpy(dst, src, bytes, hipMemcpyHostToDevice));
  return PIPO_OK;
}

pipo_status pipo_copy_d2h(void* dst, const void* src, size_t bytes) {
  clear_error();
  if (bytes) PIPO_HIP_TRY(hipMemcpy(dst, src, bytes, hipMemcpyDeviceToHost));
  return PIPO_OK;
}

pipo_status pipo_dev_synchronize(void) {
  clear_error();
  PIPO_HIP_TRY(hipDeviceSynchronize());
  return PIPO_OK;
}

static pipo_status gemm_common(GemmArgs& a, bool w4, void* out, int32_t epi, void* workspace,
                               int64_t workspace_bytes, void* stream) {
  if (((epi < 0 || epi > PIPO_EPI_F32) && epi != PIPO_EPI_SWIGLU) || !out) {
    set_error("gemm: bad epilogue %d or NULL output", epi);
    return PIPO_ERR_ARG;
  }
  if (workspace_bytes < 0) {
    set_error("gemm: negative workspace size");
    return PIPO_ERR_ARG;
  }
  a.ldo = epi == PIPO_EPI_SWIGLU ? a.N / 2 : a.N;
  if (epi == PIPO_EPI_F16 || epi == PIPO_EPI_RELU_F16 || epi == PIPO_EPI_SWIGLU)
    a.out16 = static_cast<uint16_t*>(out);
  else
    a.out32 = static_cast<float*>(out);
  return launch_gemm(a, w4, epi, static_cast<float*>(workspace), workspace ? workspace_bytes : 0,
                     static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_gemm_f16(const uint16_t* X, const uint16_t* W, const uint16_t* bias,
                             void* out, int64_t M, int64_t N, int64_t K, int32_t epi,
                             void* workspace, int64_t workspace_bytes, void* stream) {
  clear_error();
  GemmArgs a;
  a.X = X;
  a.W = W;
  a.bias = bias;
  a.M = M;
  a.N = N;
  a.K = K;
  return gemm_common(a, false, out, epi, workspace, workspace_bytes, stream);
}

pipo_status pipo_op_gemm_w4(const uint16_t* X, const uint8_t* Wq, const uint16_t* Wsm,
                            const uint16_t* bias, void* out, int64_t M, int64_t N, int64_t K,
                            int32_t epi, void* workspace, int64_t workspace_bytes, void* stream) {
  clear_error();
  GemmArgs a;
  a.X = X;
  a.Wq = Wq;
  a.Wsm = Wsm;
  a.bias = bias;
  a.M = M;
  a.N = N;
  a.K = K;
  return gemm_common(a, true, out, epi, workspace, workspace_bytes, stream);
}

pipo_status pipo_op_gemm_f16_frag(const uint16_t* X, const uint16_t* W, const uint16_t* bias,
                                  void* out, int64_t M, int64_t N, int64_t K, int32_t epi,
                                  void* workspace, int64_t workspace_bytes, void* stream) {
  clear_error();
  GemmArgs a;
  a.X = X;
  a.W = W;
  a.bias = bias;
  a.M = M;
  a.N = N;
  a.K = K;
  a.packed = true;
  return gemm_common(a, false, out, epi, workspace, workspace_bytes, stream);
}

pipo_status pipo_op_gemm_w4_frag(const uint16_t* X, const uint8_t* Wq, const uint16_t* Wsm,
                                 const uint16_t* bias, void* out, int64_t M, int64_t N,
                                 int64_t K, int32_t epi, void* workspace,
                                 int64_t workspace_bytes, void* stream) {
  clear_error();
  GemmArgs a;
  a.X = X;
  a.Wq = Wq;
  a.Wsm = Wsm;
  a.bias = bias;
  a.M = M;
  a.N = N;
  a.K = K;
  a.packed = true;
  return gemm_common(a, true, out, epi, workspace, workspace_bytes, stream);
}

int64_t pipo_op_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int32_t wfmt) {
  return gemm_workspace_bytes(M, N, K, wfmt == PIPO_W_INT4_G64);
}

pipo_status pipo_op_layernorm(const float* x, const uint16_t* gamma, const uint16_t* beta,
                              uint16_t* y, int64_t rows, int64_t d, int64_t src_stride,
                              int64_t src_offset, float eps, void* stream) {
  clear_error();
  if (!x || !gamma || !beta || !y || src_stride < 1 || src_offset < 0 || src_offset >= src_stride) {
    set_error("layernorm: bad arguments");
    return PIPO_ERR_ARG;
  }
  return launch_layernorm(x, gamma, beta, y, rows, d, src_stride, src_offset, eps,
                          static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_attn_decode(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                uint16_t* o, int32_t b, int32_t n_heads, int32_t head_dim,
                                int32_t t, void* workspace, int64_t workspace_bytes,
                                void* stream) {
  clear_error();
  if (!q || !kc || !vc || !o || workspace_bytes < 0) {
    set_error("attn_decode: NULL pointer or negative workspace size");
    return PIPO_ERR_ARG;
  }
  return launch_attn_decode(q, kc, vc, o, b, n_heads, n_heads, head_dim, t, false,
                            static_cast<float*>(workspace), workspace_bytes,
                            static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_attn_decode_kv4(const uint16_t* q, const uint8_t* kc, const uint8_t* vc,
                                    uint16_t* o, int32_t b, int32_t n_heads, int32_t head_dim,
                                    int32_t t, void* workspace, int64_t workspace_bytes,
                                    void* stream) {
  clear_error();
  if (!q || !kc || !vc || !o || workspace_bytes < 0) {
    set_error("attn_decode_kv4: NULL pointer or negative workspace size");
    return PIPO_ERR_ARG;
  }
  return launch_attn_decode(q, kc, vc, o, b, n_heads, n_heads, head_dim, t, true,
                            static_cast<float*>(workspace), workspace_bytes,
                            static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_kv_quant(const uint16_t* x, uint8_t* out, int64_t rows, int64_t d,
                             void* stream) {
  clear_error();
  if (!x || !out) {
    set_error("kv_quant: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_kv_quant(x, out, rows, d, static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_kv_dequant(const uint8_t* in, uint16_t* y, int64_t rows, int64_t d,
                               void* stream) {
  clear_error();
  if (!in || !y) {
    set_error("kv_dequant: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_kv_dequant(in, y, rows, d, static_cast<hipStream_t>(stream));
}

int64_t pipo_op_attn_decode_workspace_bytes(int32_t b, int32_t n_heads, int32_t head_dim,
                                            int32_t t) {
  if (b < 1 || n_heads < 1 || t < 0 || head_dim < 1) return 0;
  // enough for the fp16 and the INT4 cache (their workgroups differ)
  return std::max(
      attn_decode_workspace_bytes(b, n_heads, head_dim,
                                  attn_decode_splits(b, n_heads, n_heads, t, false)),
      attn_decode_workspace_bytes(b, n_heads, head_dim,
                                  attn_decode_splits(b, n_heads, n_heads, t, true)));
}

pipo_status pipo_op_attn_prefill(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                 uint16_t* o, int32_t b, int32_t P, int32_t n_heads,
                                 int32_t head_dim, void* stream) {
  clear_error();
  if (!q || !kc || !vc || !o) {
    set_error("attn_prefill: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_attn_prefill(q, kc, vc, o, b, P, n_heads, n_heads, head_dim,
                             static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_attn_decode_gqa(const uint16_t* q, const void* kc, const void* vc,
                                    uint16_t* o, int32_t b, int32_t n_heads, int32_t n_kv_heads,
                                    int32_t head_dim, int32_t t, int32_t kv_fmt, void* workspace,
                                    int64_t workspace_bytes, void* stream) {
  clear_error();
  if (!q || !kc || !vc || !o || workspace_bytes < 0 ||
      (kv_fmt != PIPO_KV_FP16 && kv_fmt != PIPO_KV_INT4_G64)) {
    set_error("attn_decode_gqa: NULL pointer, negative workspace size or unknown kv_fmt");
    return PIPO_ERR_ARG;
  }
  return launch_attn_decode(q, kc, vc, o, b, n_heads, n_kv_heads, head_dim, t,
                            kv_fmt == PIPO_KV_INT4_G64, static_cast<float*>(workspace),
                            workspace_bytes, static_cast<hipStream_t>(stream));
}

int64_t pipo_op_attn_decode_gqa_workspace_bytes(int32_t b, int32_t n_heads, int32_t n_kv_heads,
                                                int32_t head_dim, int32_t t) {
  if (b < 1 || n_heads < 1 || n_kv_heads < 1 || t < 0 || head_dim < 1) return 0;
  return std::max(
      attn_decode_workspace_bytes(b, n_heads, head_dim,
                                  attn_decode_splits(b, n_heads, n_kv_heads, t, false)),
      attn_decode_workspace_bytes(b, n_heads, head_dim,
                                  attn_decode_splits(b, n_heads, n_kv_heads, t, true)));
}

pipo_status pipo_op_attn_prefill_gqa(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                     uint16_t* o, int32_t b, int32_t P, int32_t n_heads,
                                     int32_t n_kv_heads, int32_t head_dim, void* stream) {
  clear_error();
  if (!q || !kc || !vc || !o) {
    set_error("attn_prefill_gqa: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_attn_prefill(q, kc, vc, o, b, P, n_heads, n_kv_heads, head_dim,
                             static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_rmsnorm(const float* x, const uint16_t* gamma, uint16_t* y, int64_t rows,
                            int64_t d, int64_t src_stride, int64_t src_offset, float eps,
                            void* stream) {
  clear_error();
  if (!x || !gamma || !y || src_stride < 1 || src_offset < 0 || src_offset >= src_stride) {
    set_error("rmsnorm: bad arguments");
    return PIPO_ERR_ARG;
  }
  return launch_rmsnorm(x, gamma, y, rows, d, src_stride, src_offset, eps,
                        static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_rope(uint16_t* q, uint16_t* k, const float* cos_sin, int64_t M,
                         int64_t rows_per_seq, int64_t pos0, int64_t kpos0, int64_t batch,
                         int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, float q_scale,
                         void* stream) {
  clear_error();
  if (!q || !k || !cos_sin) {
    set_error("rope: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_rope(q, k, cos_sin, M, rows_per_seq, pos0, kpos0, batch, n_heads, n_kv_heads,
                     head_dim, q_scale, static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_swiglu(const uint16_t* gu, uint16_t* h, int64_t M, int64_t F, void* stream) {
  clear_error();
  if (!gu || !h) {
    set_error("swiglu: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_swiglu(gu, h, M, F, static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_embed(const int32_t* ids, const uint16_t* tok_table, const uint16_t* pos_table,
                          float* x, int64_t rows, int64_t d, int64_t rows_per_seq, int64_t pos0,
                          int64_t pos_offset, void* stream) {
  clear_error();
  if (!ids || !tok_table || !x || rows_per_seq < 1 || pos0 < 0 || pos_offset < 0) {
    set_error("embed: bad arguments");
    return PIPO_ERR_ARG;
  }
  return launch_embed(nullptr, ids, tok_table, pos_table, x, rows, d, rows_per_seq, pos0,
                      pos_offset, static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_argmax(const float* logits, int32_t* next, int64_t rows, int64_t V,
                           void* stream) {
  clear_error();
  if (!logits || !next) {
    set_error("argmax: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_argmax(logits, next, rows, V, nullptr, 0, static_cast<hipStream_t>(stream));
}

pipo_status pipo_op_argmax_ws(const float* logits, int32_t* next, int64_t rows, int64_t V,
                              void* workspace, int64_t workspace_bytes, void* stream) {
  clear_error();
  if (!logits || !next || workspace_bytes < 0) {
    set_error("argmax: NULL pointer or negative workspace size");
    return PIPO_ERR_ARG;
  }
  return launch_argmax(logits, next, rows, V, workspace, workspace ? workspace_bytes : 0,
                       static_cast<hipStream_t>(stream));
}

int64_t pipo_op_argmax_workspace_bytes(int64_t rows, int64_t V) {
  if (rows < 1 || V < 1) return 0;
  return argmax_workspace_bytes(rows, V);
}

pipo_status pipo_op_copy(void* dst, const void* src, int64_t bytes, void* stream) {
  clear_error();
  if (!dst || !src) {
    set_error("copy: NULL pointer");
    return PIPO_ERR_ARG;
  }
  return launch_copy16(dst, src, bytes, static_cast<hipStream_t>(stream));
}

}  // extern "C"
