/*
 * pipo_sched.h -- the pipeline schedule as data, for checking it without a
 * GPU.  The library's engine executes exactly these operation lists on HIP
 * streams; this entry point returns them as text instead.
 *
 * The schedule is PIPO's pipeline scheduling (Algorithm 1, Section 3.2.2):
 * per unit (a layer, or the output head), load its weights ahead of time
 * into a rotating HBM slot, synchronise each kernel on the load of the
 * tensor it reads, compute, and -- with the KV cache in host memory -- load
 * each layer's cache prefix before its attention and save the new rows
 * after the QKV projection.
 */
#ifndef PIPO_SCHED_H
#define PIPO_SCHED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_layers;
  int32_t n_slots;          /* >= 1 (1: no unit is loaded before the previous one is done) */
  int32_t n_h2d;            /* 1 or 2 */
  int32_t layers_streamed;  /* 0/1 */
  int32_t head_streamed;    /* 0/1 */
  int32_t kv_on_host;       /* 0/1 (requires layers_streamed) */
  int32_t poison;           /* 0/1 */
  int32_t delay;            /* 0/1 */
  int64_t chunk_bytes;      /* > 0 */
  int64_t layer_seg_bytes[10]; /* bytes of the 10 segments of a layer unit (head entry unused) */
  int64_t head_bytes;
  int32_t merged;           /* 0/1: copy a layer's matrix segments (1..8) as one byte range
                               from segment 1's slot offset, in chunks that may span
                               segments; segment 0 is copied alone */
  int64_t layer_seg_off[10]; /* slot offsets of the segments (used when merged) */
} pipo_sched_config;

/*
 * Generate the operations of n_passes consecutive passes (pass i: prefill
 * if prefill[i], appending T[i] positions at pos0[i], KV rows of
 * kv_row_bytes each) and write them to buf (host, buflen bytes), one per
 * line as eleven integers:
 *   kind stream event kernel unit layer slot seg kv off bytes
 * kind: 0 copy-h2d, 1 copy-d2h, 2 wait, 3 record, 4 kernel, 5 delay,
 *       6 poison, 7 readback;  stream: 0 compute, 1-2 h2d, 3 d2h;
 * kernel: 0 embed, 1 ln1, 2 qkv, 3 attn, 4 oproj, 5 ln2, 6 fc1, 7 fc2,
 *         8 lnf, 9 head, 10 argmax.  A merged weight copy names segment 1;
 * its off counts from that segment's slot offset.
 * Returns the number of bytes written (excluding the final NUL), or -1 if
 * the arguments are invalid or buf is too small.
 */
int64_t pipo_sched_trace(const pipo_sched_config* cfg, int32_t n_passes, const int32_t* prefill,
                         const int64_t* pos0, const int64_t* T, int64_t kv_row_bytes, char* buf,
                         int64_t buflen);

#ifdef __cplusplus
}
#endif

#endif /* PIPO_SCHED_H */
