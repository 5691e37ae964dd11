// Memory planning and the automatic configuration (Section 3.5, Eq. (1),
// and Algorithm 2's Configure step), re-derived for this implementation:
// instead of the paper's closed forms for LLaMA (Appendix B), the footprint
// of a policy is the exact sum of what pipo_create allocates (plan.h).
#include <unistd.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "plan.h"

namespace pipo {

pipo_status check_shape(const pipo_shape* s) {
  if (!s) {
    set_error("shape is NULL");
    return PIPO_ERR_ARG;
  }
  if (s->n_layers < 1 || s->d_model < 1 || s->n_heads < 1 || s->d_ffn < 1 || s->vocab < 1 ||
      s->max_pos < 1 || s->pos_offset < 0 || !(s->ln_eps >= 0.f)) {
    set_error("invalid shape");
    return PIPO_ERR_ARG;
  }
  if (s->d_model % s->n_heads != 0) {
    set_error("d_model %d is not a multiple of n_heads %d", s->d_model, s->n_heads);
    return PIPO_ERR_ARG;
  }
  const int dh = s->d_model / s->n_heads;
  if (dh != 64 && dh != 128) {
    set_error("head_dim %d not supported (64 or 128)", dh);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (s->d_model % 128 != 0 || s->d_ffn % 128 != 0 || s->d_model > 8192) {
    set_error("d_model %d / d_ffn %d must be multiples of 128 (d_model <= 8192)", s->d_model,
              s->d_ffn);
    return PIPO_ERR_UNSUPPORTED;
  }
  return PIPO_OK;
}

pipo_status normalize_policy(const pipo_shape* shape, pipo_policy* p) {
  pipo_policy& pol = *p;
  if (pol.wfmt != PIPO_W_FP16 && pol.wfmt != PIPO_W_INT4_G64) {
    set_error("unknown weight format %d", pol.wfmt);
    return PIPO_ERR_ARG;
  }
  if (pol.n_weight_slots == 0) pol.n_weight_slots = 3;
  if (pol.n_h2d_streams == 0) pol.n_h2d_streams = 2;
  if (pol.chunk_bytes == 0) pol.chunk_bytes = 64ll << 20;
  pol.chunk_bytes = align_up(pol.chunk_bytes, 4096);
  if (pol.n_weight_slots < 1 || pol.n_weight_slots > 16 || pol.n_h2d_streams < 1 ||
      pol.n_h2d_streams > 2 || pol.max_batch < 1 || pol.max_seq < 1 || pol.chunk_bytes < 0 ||
      pol.copy_delay_us < 0) {
    set_error("invalid policy");
    return PIPO_ERR_ARG;
  }
  if (pol.max_seq > shape->max_pos || pol.max_seq > kAttnDecodeMaxT) {
    set_error("max_seq %d exceeds max_pos %d or the decode kernel's %d keys", pol.max_seq,
              shape->max_pos, kAttnDecodeMaxT);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (pol.kv_on_host && !pol.weights_on_host) {
    set_error("kv_on_host requires weights_on_host");
    return PIPO_ERR_UNSUPPORTED;
  }
  if (pol.kv_fmt != PIPO_KV_FP16 && pol.kv_fmt != PIPO_KV_INT4_G64) {
    set_error("unknown kv_fmt %d", pol.kv_fmt);
    return PIPO_ERR_ARG;
  }
  if (pol.kv_fmt == PIPO_KV_INT4_G64 && shape->d_model % 256 != 0) {
    set_error("an INT4 KV cache needs d_model %% 256 == 0 (d_model=%d)", shape->d_model);
    return PIPO_ERR_UNSUPPORTED;
  }
  return PIPO_OK;
}

UnitLayout unit_layout(const pipo_shape& sh, bool w4) {
  UnitLayout u;
  const int64_t d = sh.d_model, F = sh.d_ffn, V = sh.vocab;
  u.misc_bytes = (9 * d + F) * 2;
  const auto mat = [&](int seg, int64_t N, int64_t K) {
    if (w4) {
      u.seg_bytes[seg] = N * K / 2;
      u.seg_bytes[seg + 1] = N * (K / 64) * 4;
    } else {
      u.seg_bytes[seg] = N * K * 2;
    }
  };
  u.seg_bytes[kSegMisc] = u.misc_bytes;
  mat(kSegWqkv, 3 * d, d);
  mat(kSegWo, d, d);
  mat(kSegW1, F, d);
  mat(kSegW2, d, F);
  int64_t off = 0;
  for (int sg = 0; sg < kNumSegs; ++sg) {
    if (sg == kSegHead) continue;
    u.seg_off[sg] = off;
    off = align_up(off + u.seg_bytes[sg], 4096);
    u.copy_bytes += u.seg_bytes[sg];
  }
  u.layer_bytes = off;
  u.head_bytes = V * d * 2;
  return u;
}

HbmPlan hbm_plan(const pipo_shape& sh, const pipo_policy& pol) {
  HbmPlan p;
  const bool w4 = pol.wfmt == PIPO_W_INT4_G64, kv4 = pol.kv_fmt == PIPO_KV_INT4_G64;
  const UnitLayout u = unit_layout(sh, w4);
  const int64_t d = sh.d_model, F = sh.d_ffn, V = sh.vocab, L = sh.n_layers;
  const int64_t rows = (int64_t)pol.max_batch * pol.max_seq;
  if (pol.weights_on_host) p.slot_bytes = u.layer_bytes;
  if (pol.embed_on_host) p.slot_bytes = std::max(p.slot_bytes, align_up(u.head_bytes, 4096));
  p.slots = p.slot_bytes * pol.n_weight_slots;
  p.resident = pol.weights_on_host ? 0 : u.layer_bytes * L;
  p.tok = pol.embed_on_host ? 0 : u.head_bytes;
  p.pos = ((int64_t)sh.max_pos + sh.pos_offset) * d * 2;
  p.lnf = d * 4;
  p.x = rows * d * 4;
  p.a = rows * d * 2;
  p.q = rows * d * 2;
  p.o = rows * d * 2;
  p.h = rows * F * 2;
  p.logits = (int64_t)pol.max_batch * V * 4;
  p.next = (int64_t)pol.max_batch * 4;
  p.ids = rows * 4;
  p.emb = pol.embed_on_host ? rows * d * 2 : 0;
  p.attn_ws = attn_decode_workspace_bytes(pol.max_batch, sh.n_heads, (int)(d / sh.n_heads),
                                          kAttnDecodeMaxSplits);
  const int64_t shapes[5][3] = {{3 * d, d, w4}, {d, d, w4}, {F, d, w4}, {d, F, w4}, {V, d, 0}};
  for (const auto& s : shapes)
    p.gemm_ws = std::max(p.gemm_ws, gemm_workspace_bytes_upto(rows, s[0], s[1], s[2] != 0));
  p.kstage = kv4 ? rows * d * 2 : 0;
  p.kv_row = kv4 ? d / 2 + d / 16 : 2 * d;
  p.kv_part = rows * p.kv_row;
  p.kv = (pol.kv_on_host ? pol.n_weight_slots : L) * 2 * p.kv_part;
  return p;
}

int64_t host_kv_bytes(const pipo_shape& sh, const pipo_policy& pol) {
  if (!pol.kv_on_host) return 0;
  const HbmPlan p = hbm_plan(sh, pol);
  return (int64_t)sh.n_layers * align_up(2 * p.kv_part, 4096);
}

// bytes one decode step moves host -> device at the last position
static int64_t step_bytes(const pipo_shape& sh, const pipo_policy& pol) {
  const UnitLayout u = unit_layout(sh, pol.wfmt == PIPO_W_INT4_G64);
  const HbmPlan p = hbm_plan(sh, pol);
  const int64_t b = pol.max_batch, d = sh.d_model, t = pol.max_seq - 1;
  int64_t bytes = b * 4;  // token ids
  if (pol.weights_on_host) bytes += (int64_t)sh.n_layers * u.copy_bytes;
  if (pol.embed_on_host) bytes += u.head_bytes + b * d * 2;
  if (pol.kv_on_host) bytes += (int64_t)sh.n_layers * 2 * t * b * p.kv_row;
  return bytes;
}

static void fill_plan(const pipo_shape& sh, const pipo_policy& pol, pipo_plan* out) {
  const UnitLayout u = unit_layout(sh, pol.wfmt == PIPO_W_INT4_G64);
  const HbmPlan p = hbm_plan(sh, pol);
  std::memset(out, 0, sizeof *out);
  out->weight_bytes = (int64_t)sh.n_layers * u.copy_bytes + u.head_bytes +
                      ((int64_t)sh.max_pos + sh.pos_offset) * sh.d_model * 2 + 4 * sh.d_model;
  out->kv_bytes = (int64_t)sh.n_layers * 2 * p.kv_part;
  out->hbm_bytes = p.total();
  out->host_kv_bytes = host_kv_bytes(sh, pol);
  out->h2d_bytes_per_step = step_bytes(sh, pol);
  out->pipeline = pol.n_weight_slots >= 2 ? PIPO_PIPE_PERFORMANCE : PIPO_PIPE_MEMORY_EFFICIENT;
}

}  // namespace pipo

using namespace pipo;

extern "C" {

pipo_status pipo_plan_policy(const pipo_shape* shape, const pipo_policy* policy,
                             pipo_plan* plan_out) {
  clear_error();
  PIPO_TRY(check_shape(shape));
  if (!policy || !plan_out) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  pipo_policy pol = *policy;
  PIPO_TRY(normalize_policy(shape, &pol));
  fill_plan(*shape, pol, plan_out);
  return PIPO_OK;
}

pipo_status pipo_configure(const pipo_shape* shape, int32_t wfmt, int32_t kv_fmt,
                           int32_t max_batch, int32_t max_seq, const pipo_resources* res,
                           pipo_policy* policy_out, pipo_plan* plan_out) {
  clear_error();
  PIPO_TRY(check_shape(shape));
  if (!res || !policy_out) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  int64_t hbm = res->hbm_bytes, host = res->host_bytes;
  if (hbm < 0 || host < 0) {
    set_error("negative resource size");
    return PIPO_ERR_ARG;
  }
  if (hbm == 0) {
    size_t free_b = 0, total_b = 0;
    PIPO_HIP_TRY(hipMemGetInfo(&free_b, &total_b));
    hbm = (int64_t)free_b;
  }
  if (host == 0) host = (int64_t)sysconf(_SC_AVPHYS_PAGES) * (int64_t)sysconf(_SC_PAGESIZE);

  // Eq. (1) generalised: among the placements that fit (weights and head
  // resident or streamed, KV resident or in host memory) and the two
  // pipelines, take the one that streams the fewest bytes per decode step;
  // at equal bytes, the performance-optimized pipeline (more slots).
  pipo_policy best{};
  int64_t best_bytes = -1, best_slots = 0, need_hbm = -1, need_host = -1;
  pipo_status first_err = PIPO_OK;
  for (int w_host = 0; w_host <= 1; ++w_host)
    for (int e_host = 0; e_host <= 1; ++e_host)
      for (int kv_host = 0; kv_host <= w_host; ++kv_host)
        for (int slots : {3, 2, 1}) {
          if (!w_host && !e_host && slots != 3) continue;  // nothing streams: slots unused
          pipo_policy pol{};
          pol.wfmt = wfmt;
          pol.kv_fmt = kv_fmt;
          pol.weights_on_host = w_host;
          pol.embed_on_host = e_host;
          pol.kv_on_host = kv_host;
          pol.n_weight_slots = slots;
          pol.max_batch = max_batch;
          pol.max_seq = max_seq;
          const pipo_status st = normalize_policy(shape, &pol);
          if (st != PIPO_OK) {
            if (first_err == PIPO_OK) first_err = st;
            continue;
          }
          const int64_t h = hbm_plan(*shape, pol).total();
          const int64_t k = host_kv_bytes(*shape, pol);
          if (need_hbm < 0 || h < need_hbm) need_hbm = h;
          if (h > hbm) continue;
          if (need_host < 0 || k < need_host) need_host = k;  // among those that fit in HBM
          if (k > host) continue;
          const int64_t bytes = step_bytes(*shape, pol);
          if (best_bytes < 0 || bytes < best_bytes || (bytes == best_bytes && slots > best_slots)) {
            best = pol;
            best_bytes = bytes;
            best_slots = slots;
          }
        }
  if (best_bytes < 0) {
    if (first_err != PIPO_OK && need_hbm < 0) return first_err;
    if (need_host < 0) {
      set_error("even the memory-efficient pipeline needs %lld bytes of HBM (%lld available)",
                (long long)need_hbm, (long long)hbm);
      return PIPO_ERR_OOM_DEVICE;
    }
    set_error("the KV cache needs %lld bytes of host memory (%lld available); a disk tier "
              "would be needed, which this library does not have",
              (long long)need_host, (long long)host);
    return PIPO_ERR_OOM_HOST;
  }
  best.hbm_budget_bytes = hbm;
  *policy_out = best;
  if (plan_out) fill_plan(*shape, best, plan_out);
  return PIPO_OK;
}

}  // extern "C"
