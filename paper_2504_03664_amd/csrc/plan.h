// What pipo_create allocates, computed without allocating anything.  The
// context, pipo_plan_policy and pipo_configure all size memory through
// these functions, so a planned footprint is the real one.
#pragma once

#include "common.h"
#include "schedule.h"

namespace pipo {

inline int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

pipo_status check_shape(const pipo_shape* s);

inline bool is_llama(const pipo_shape& s) { return s.family == PIPO_FAMILY_LLAMA; }
inline int64_t kv_heads(const pipo_shape& s) { return s.n_kv_heads > 0 ? s.n_kv_heads : s.n_heads; }
// width of a cached key (value) row: n_kv_heads * head_dim
inline int64_t kv_width(const pipo_shape& s) { return kv_heads(s) * (s.d_model / s.n_heads); }
// output rows of the fused QKV matrix and of the first MLP matrix
inline int64_t qkv_rows(const pipo_shape& s) { return s.d_model + 2 * kv_width(s); }
inline int64_t fc1_rows(const pipo_shape& s) { return is_llama(s) ? 2 * (int64_t)s.d_ffn : s.d_ffn; }

// (cos, sin) of p * w_i for p < n_pos, i < head_dim / 2 (rotary positions)
void rope_table(const pipo_shape& s, int64_t n_pos, float* out);

// defaults (0 fields) and range checks of a policy, in place
pipo_status normalize_policy(const pipo_shape* shape, pipo_policy* pol);

// small tensors of a layer, packed in this order (absent ones take no room)
enum MiscTensor { kLn1G, kLn1B, kBqkv, kBo, kLn2G, kLn2B, kB1, kB2, kNumMisc };
// shortest host-to-device copy that the runtime gives to a DMA engine
constexpr int64_t kMinDmaCopyBytes = 32768;

// one layer unit as it sits in a weight slot: segments at 4 KiB offsets
struct UnitLayout {
  int64_t seg_bytes[kNumSegs] = {};
  int64_t seg_off[kNumSegs] = {};
  int64_t misc_count[kNumMisc] = {};  // elements (0: absent)
  int64_t misc_off[kNumMisc] = {};    // element offsets in the packed block
  int64_t misc_bytes = 0;    // small tensors of a layer, packed
  int64_t layer_bytes = 0;   // slot bytes of a layer unit
  int64_t copy_bytes = 0;    // bytes a layer unit's copies move (sum of segments)
  int64_t tensor_bytes = 0;  // bytes of a layer's tensors (copy_bytes without the padding
                             // of the small-tensor copy to kMinDmaCopyBytes)
  int64_t head_bytes = 0;    // the output head (the token table when tied)
};
UnitLayout unit_layout(const pipo_shape& sh, bool w4);

// every device allocation of a context (bytes; 0 where not allocated)
struct HbmPlan {
  int64_t slot_bytes = 0, slots = 0, resident = 0, tok = 0, head = 0, pos = 0, lnf = 0;
  int64_t x = 0, a = 0, q = 0, o = 0, h = 0, gu = 0, logits = 0, next = 0, ids = 0, emb = 0;
  int64_t rope = 0;                              // rotary (cos, sin) table
  int64_t attn_ws = 0, gemm_ws = 0, argmax_ws = 0;
  int64_t kstage = 0;                            // each of the K and V staging buffers
  int64_t kv_row = 0, kv_part = 0, kv = 0;
  int64_t total() const {
    return slots + resident + tok + head + pos + lnf + x + a + q + o + h + gu + logits + next +
           ids + emb + rope + attn_ws + gemm_ws + argmax_ws + 2 * kstage + kv;
  }
};
HbmPlan hbm_plan(const pipo_shape& sh, const pipo_policy& pol);  // pol normalized

// host memory the library allocates for the KV cache (per layer, 4 KiB aligned)
int64_t host_kv_bytes(const pipo_shape& sh, const pipo_policy& pol);

// pinned staging rings (pageable host KV layers, disk tier) and the disk
// tier's pageable direct-I/O chunk: buffers of chunk_bytes
constexpr int kStageH2DBufs = 16, kStageD2HBufs = 8;
int64_t staging_bytes(const pipo_policy& pol);

// weights kept in host memory (streamed layers unless on disk, streamed head)
// plus the staging rings
int64_t host_weight_bytes(const pipo_shape& sh, const pipo_policy& pol);

// the disk tier's file: every layer unit in slot layout
int64_t disk_file_bytes(const pipo_shape& sh, const pipo_policy& pol);

}  // namespace pipo
