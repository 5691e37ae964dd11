// Memory planning and the automatic configuration (Section 3.5, Eq. (1),
// and Algorithm 2's Configure step), re-derived for this implementation:
// instead of the paper's closed forms for LLaMA (Appendix B), the footprint
// of a policy is the exact sum of what pipo_create allocates (plan.h).
#include <unistd.h>

#include <algorithm>
#include <cmath>
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
  if (s->family != PIPO_FAMILY_OPT && s->family != PIPO_FAMILY_LLAMA) {
    set_error("unknown model family %d", s->family);
    return PIPO_ERR_ARG;
  }
  const int hkv = (int)kv_heads(*s);
  if (s->n_kv_heads < 0 || s->n_heads % hkv != 0) {
    set_error("n_heads %d is not a multiple of n_kv_heads %d", s->n_heads, s->n_kv_heads);
    return PIPO_ERR_ARG;
  }
  const int group = s->n_heads / hkv;
  if (group != 1 && group != 2 && group != 4 && group != 8) {
    set_error("%d query heads per key/value head not supported (1, 2, 4, 8)", group);
    return PIPO_ERR_UNSUPPORTED;
  }
  if (s->family == PIPO_FAMILY_OPT && group != 1) {
    set_error("the OPT family has no grouped-query attention (n_kv_heads %d)", s->n_kv_heads);
    return PIPO_ERR_ARG;
  }
  if (s->family == PIPO_FAMILY_LLAMA) {
    if (!(s->rope_theta > 0.f) || !(s->rope_factor >= 0.f)) {
      set_error("invalid rotary base %g or scaling factor %g", (double)s->rope_theta,
                (double)s->rope_factor);
      return PIPO_ERR_ARG;
    }
    if (s->rope_factor > 0.f &&
        !(s->rope_low_freq_factor > 0.f && s->rope_high_freq_factor > s->rope_low_freq_factor &&
          s->rope_orig_max_pos > 0)) {
      set_error("invalid rotary scaling: low %g, high %g, original length %d",
                (double)s->rope_low_freq_factor, (double)s->rope_high_freq_factor,
                s->rope_orig_max_pos);
      return PIPO_ERR_ARG;
    }
  }
  return PIPO_OK;
}

// Rotary angles (the LLaMA 3.1 reading of the family): w_i = theta^(-2i/D);
// with scaling, a wavelength 2 pi / w above orig / low is divided by the
// factor, one below orig / high is kept, and in between the two are blended
// linearly in orig / wavelength.  Angles and their sines in double.
void rope_table(const pipo_shape& s, int64_t n_pos, float* out) {
  const int D = s.d_model / s.n_heads, half = D / 2;
  std::vector<double> w((size_t)half);
  for (int i = 0; i < half; ++i) {
    double wi = std::pow((double)s.rope_theta, -2.0 * i / D);
    if (s.rope_factor > 0.f) {
      const double factor = s.rope_factor, lo = s.rope_low_freq_factor,
                   hi = s.rope_high_freq_factor, orig = s.rope_orig_max_pos;
      const double wavelen = 2.0 * M_PI / wi;
      if (wavelen > orig / lo) {
        wi /= factor;
      } else if (wavelen >= orig / hi) {
        const double sm = (orig / wavelen - lo) / (hi - lo);
        wi = (1.0 - sm) * wi / factor + sm * wi;
      }
    }
    w[(size_t)i] = wi;
  }
  for (int64_t p = 0; p < n_pos; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)p * w[(size_t)i];
      out[(p * half + i) * 2] = (float)std::cos(ang);
      out[(p * half + i) * 2 + 1] = (float)std::sin(ang);
    }
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
  if (pol.weights_on_disk && !pol.weights_on_host) {
    set_error("weights_on_disk requires weights_on_host (the layers stream every pass)");
    return PIPO_ERR_UNSUPPORTED;
  }
  if (pol.copy_threads < 0 || pol.copy_threads > 64) {
    set_error("copy_threads %d outside [0, 64]", pol.copy_threads);
    return PIPO_ERR_ARG;
  }
  if (pol.kv_fmt != PIPO_KV_FP16 && pol.kv_fmt != PIPO_KV_INT4_G64) {
    set_error("unknown kv_fmt %d", pol.kv_fmt);
    return PIPO_ERR_ARG;
  }
  if (pol.kv_fmt == PIPO_KV_INT4_G64 && kv_width(*shape) % 256 != 0) {
    set_error("an INT4 KV cache needs rows of a multiple of 256 elements (%lld)",
              (long long)kv_width(*shape));
    return PIPO_ERR_UNSUPPORTED;
  }
  return PIPO_OK;
}

UnitLayout unit_layout(const pipo_shape& sh, bool w4) {
  UnitLayout u;
  const int64_t d = sh.d_model, F = sh.d_ffn, V = sh.vocab;
  if (is_llama(sh)) {
    u.misc_count[kLn1G] = d;
    u.misc_count[kLn2G] = d;
  } else {
    const int64_t cnt[kNumMisc] = {d, d, 3 * d, d, d, d, F, d};
    for (int i = 0; i < kNumMisc; ++i) u.misc_count[i] = cnt[i];
  }
  int64_t elems = 0;
  for (int i = 0; i < kNumMisc; ++i) {
    u.misc_off[i] = elems;
    elems += u.misc_count[i];
  }
  u.misc_bytes = elems * 2;
  const auto mat = [&](int seg, int64_t N, int64_t K) {
    if (w4) {
      u.seg_bytes[seg] = N * K / 2;
      u.seg_bytes[seg + 1] = N * (K / 64) * 4;
    } else {
      u.seg_bytes[seg] = N * K * 2;
    }
  };
  // The small tensors are copied on their own; a host-to-device copy
  // shorter than 32 KiB is served by a blit kernel on the compute units
  // instead of a DMA engine (measured: 16 KiB copies run
  // __amd_rocclr_copyBuffer, 32 KiB ones do not), so that copy is padded to
  // kMinDmaCopyBytes (zeros beyond the last layer's tensors).
  u.seg_bytes[kSegMisc] = std::max(u.misc_bytes, kMinDmaCopyBytes);
  mat(kSegWqkv, qkv_rows(sh), d);
  mat(kSegWo, d, d);
  mat(kSegW1, fc1_rows(sh), d);
  mat(kSegW2, d, F);
  int64_t off = 0;
  for (int sg = 0; sg < kNumSegs; ++sg) {
    if (sg == kSegHead) continue;
    u.seg_off[sg] = off;
    off = align_up(off + u.seg_bytes[sg], 4096);
    u.copy_bytes += u.seg_bytes[sg];
  }
  u.tensor_bytes = u.copy_bytes - (u.seg_bytes[kSegMisc] - u.misc_bytes);
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
  const bool llama = is_llama(sh);
  p.head = llama && !pol.embed_on_host ? u.head_bytes : 0;  // untied head
  p.pos = llama ? 0 : ((int64_t)sh.max_pos + sh.pos_offset) * d * 2;
  p.rope = llama ? (int64_t)pol.max_seq * (d / sh.n_heads) * 4 : 0;
  p.lnf = d * 4;
  p.x = rows * d * 4;
  p.a = rows * d * 2;
  p.q = rows * d * 2;
  p.o = rows * d * 2;
  p.h = rows * F * 2;
  p.gu = llama ? rows * 2 * F * 2 : 0;  // gate and up outputs before SwiGLU
  p.logits = (int64_t)pol.max_batch * V * 4;
  p.next = (int64_t)pol.max_batch * 4;
  p.ids = rows * 4;
  p.emb = pol.embed_on_host ? rows * d * 2 : 0;
  p.argmax_ws = argmax_workspace_bytes(pol.max_batch, V);
  p.attn_ws = attn_decode_workspace_bytes(pol.max_batch, sh.n_heads, (int)(d / sh.n_heads),
                                          kAttnDecodeMaxSplits);
  const int64_t shapes[5][3] = {
      {qkv_rows(sh), d, w4}, {d, d, w4}, {fc1_rows(sh), d, w4}, {d, F, w4}, {V, d, 0}};
  for (const auto& s : shapes)
    p.gemm_ws = std::max(p.gemm_ws, gemm_workspace_bytes_upto(rows, s[0], s[1], s[2] != 0));
  const int64_t dkv = kv_width(sh);
  // INT4 cache: new rows are staged in fp16 (and rotated there) before quantization
  p.kstage = kv4 ? rows * dkv * 2 : 0;
  p.kv_row = kv4 ? dkv / 2 + dkv / 16 : 2 * dkv;
  p.kv_part = rows * p.kv_row;
  p.kv = (pol.kv_on_host ? pol.n_weight_slots : L) * 2 * p.kv_part;
  return p;
}

int64_t host_kv_bytes(const pipo_shape& sh, const pipo_policy& pol) {
  if (!pol.kv_on_host) return 0;
  const HbmPlan p = hbm_plan(sh, pol);
  return (int64_t)sh.n_layers * align_up(2 * p.kv_part, 4096);
}

int64_t staging_bytes(const pipo_policy& pol) {
  int64_t n = 0;
  if (pol.kv_on_host || pol.weights_on_disk) n += kStageH2DBufs;
  if (pol.kv_on_host) n += kStageD2HBufs;
  if (pol.weights_on_disk) n += 1;  // the pageable chunk direct I/O goes through
  return n * pol.chunk_bytes;
}

int64_t host_weight_bytes(const pipo_shape& sh, const pipo_policy& pol) {
  const UnitLayout u = unit_layout(sh, pol.wfmt == PIPO_W_INT4_G64);
  int64_t bytes = staging_bytes(pol);
  if (pol.weights_on_host && !pol.weights_on_disk) bytes += (int64_t)sh.n_layers * u.tensor_bytes;
  if (pol.embed_on_host) bytes += u.head_bytes;
  return bytes;
}

int64_t disk_file_bytes(const pipo_shape& sh, const pipo_policy& pol) {
  if (!pol.weights_on_disk) return 0;
  return (int64_t)sh.n_layers * unit_layout(sh, pol.wfmt == PIPO_W_INT4_G64).layer_bytes;
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
  out->weight_bytes =
      (int64_t)sh.n_layers * u.tensor_bytes + u.head_bytes +
      (is_llama(sh) ? u.head_bytes + 2 * sh.d_model
                    : ((int64_t)sh.max_pos + sh.pos_offset) * sh.d_model * 2 + 4 * sh.d_model);
  out->kv_bytes = (int64_t)sh.n_layers * 2 * p.kv_part;
  out->hbm_bytes = p.total();
  out->host_kv_bytes = host_kv_bytes(sh, pol);
  out->h2d_bytes_per_step = step_bytes(sh, pol);
  out->pipeline = pol.n_weight_slots >= 2 ? PIPO_PIPE_PERFORMANCE : PIPO_PIPE_MEMORY_EFFICIENT;
  out->host_weight_bytes = host_weight_bytes(sh, pol);
  out->disk_bytes = disk_file_bytes(sh, pol);
  // each layer unit is read whole (4 KiB-aligned pieces) once per pass
  out->disk_bytes_per_step = out->disk_bytes;
}

}  // namespace pipo

using namespace pipo;

extern "C" {

pipo_status pipo_rope_table(const pipo_shape* shape, int32_t n_pos, float* out) {
  clear_error();
  PIPO_TRY(check_shape(shape));
  if (!out || n_pos < 0 || shape->family != PIPO_FAMILY_LLAMA) {
    set_error("rope_table: NULL output, negative n_pos or not a LLaMA shape");
    return PIPO_ERR_ARG;
  }
  return guarded([&] {
    rope_table(*shape, n_pos, out);
    return PIPO_OK;
  });
}

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
  int64_t hbm = res->hbm_bytes, host = res->host_bytes, disk = res->disk_bytes;
  if (hbm < 0 || host < 0 || disk < 0) {
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
  // resident or streamed, streamed layers in host memory or on disk, KV
  // resident or in host memory) and the two pipelines, take the one that
  // streams the fewest bytes per decode step; at equal bytes host memory
  // before disk, then the performance-optimized pipeline (more slots).
  pipo_policy best{};
  int64_t best_bytes = -1, best_slots = 0, need_hbm = -1, need_host = -1;
  int best_disk = 0;
  pipo_status first_err = PIPO_OK;
  for (int w_host = 0; w_host <= 1; ++w_host)
    for (int on_disk = 0; on_disk <= (w_host && disk > 0 ? 1 : 0); ++on_disk)
      for (int e_host = 0; e_host <= 1; ++e_host)
        for (int kv_host = 0; kv_host <= w_host; ++kv_host)
          for (int slots : {3, 2, 1}) {
            if (!w_host && !e_host && slots != 3) continue;  // nothing streams: slots unused
            pipo_policy pol{};
            pol.wfmt = wfmt;
            pol.kv_fmt = kv_fmt;
            pol.weights_on_host = w_host;
            pol.weights_on_disk = on_disk;
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
            const int64_t k = host_kv_bytes(*shape, pol) + host_weight_bytes(*shape, pol);
            if (need_hbm < 0 || h < need_hbm) need_hbm = h;
            if (h > hbm) continue;
            if (need_host < 0 || k < need_host) need_host = k;  // among those that fit in HBM
            if (k > host || disk_file_bytes(*shape, pol) > disk) continue;
            const int64_t bytes = step_bytes(*shape, pol);
            const bool better =
                best_bytes < 0 || bytes < best_bytes ||
                (bytes == best_bytes &&
                 (on_disk < best_disk || (on_disk == best_disk && slots > best_slots)));
            if (better) {
              best = pol;
              best_bytes = bytes;
              best_slots = slots;
              best_disk = on_disk;
            }
          }
  if (best_bytes < 0) {
    if (first_err != PIPO_OK && need_hbm < 0) return first_err;
    if (need_host < 0) {
      set_error("even the memory-efficient pipeline needs %lld bytes of HBM (%lld available)",
                (long long)need_hbm, (long long)hbm);
      return PIPO_ERR_OOM_DEVICE;
    }
    set_error("%lld bytes must stay in host memory (%lld available) even with the layers on "
              "disk (%lld bytes of disk allowed)",
              (long long)need_host, (long long)host, (long long)disk);
    return PIPO_ERR_OOM_HOST;
  }
  best.hbm_budget_bytes = hbm;
  *policy_out = best;
  if (plan_out) fill_plan(*shape, best, plan_out);
  return PIPO_OK;
}

}  // extern "C"
