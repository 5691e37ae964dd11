// Pipeline schedule generator (see schedule.h).
#include "schedule.h"

#include <algorithm>
#include <cstdio>

namespace pipo {

Scheduler::Scheduler(const SchedConfig& c) : cfg_(c) {
  ev_.n_slots = c.n_slots;
  ev_.n_layers = c.n_layers;
  U_ = (c.layers_streamed ? c.n_layers : 0) + (c.head_streamed ? 1 : 0);
  la_ = c.n_slots - 1;
  // a KV load waits on the previous token's save of its layer, recorded one
  // pass (U_ units) earlier: it must already have been issued
  if (c.kv_on_host) la_ = std::min(la_, U_ - 1);
  if (la_ < 0) la_ = 0;
  seg_streams_.assign((size_t)c.n_slots * kNumSegs, 0);
  kv_streams_.assign((size_t)c.n_slots, 0);
}

static Op make(OpKind k, int stream) {
  Op o;
  o.kind = k;
  o.stream = stream;
  return o;
}

void Scheduler::issue_weights(int64_t g, std::vector<Op>& out) {
  const int s = (int)(g % cfg_.n_slots);
  const int u = (int)(g % U_);
  const int layer = unit_layer(u);
  const int n = cfg_.n_h2d;
  if (g >= cfg_.n_slots) {
    for (int i = 0; i < n; ++i) {
      Op w = make(OpKind::Wait, kH2D0 + i);
      w.event = ev_.slot_free(s);
      w.unit = g;
      w.slot = s;
      out.push_back(w);
    }
  }
  if (cfg_.poison) {
    Op p = make(OpKind::Poison, kH2D0);
    p.unit = g;
    p.slot = s;
    out.push_back(p);
    if (n > 1) {
      Op r = make(OpKind::Record, kH2D0);
      r.event = ev_.poisoned(s);
      out.push_back(r);
      Op w = make(OpKind::Wait, kH2D1);
      w.event = ev_.poisoned(s);
      out.push_back(w);
    }
  }
  int chunk_no = 0;
  const auto seg_bytes = [&](int seg) -> int64_t {
    return layer >= 0 ? (seg == kSegHead ? 0 : cfg_.layer_seg_bytes[seg])
                      : (seg == kSegHead ? cfg_.head_bytes : 0);
  };
  const auto copy = [&](int seg, int64_t off, int64_t bytes) {
    const int st = chunk_no++ % n;
    if (cfg_.delay) out.push_back(make(OpKind::Delay, kH2D0 + st));
    Op c = make(OpKind::CopyH2D, kH2D0 + st);
    c.unit = g;
    c.layer = layer;
    c.slot = s;
    c.seg = seg;
    c.off = off;
    c.bytes = bytes;
    out.push_back(c);
    return st;
  };
  // ready events of a segment, on every stream that carried part of it
  const auto record = [&](int seg) {
    const uint8_t mask = seg_streams_[(size_t)s * kNumSegs + seg];
    for (int st = 0; st < n; ++st) {
      if (!(mask & (1u << st))) continue;
      Op r = make(OpKind::Record, kH2D0 + st);
      r.event = ev_.seg_ready(s, seg, st);
      r.unit = g;
      r.slot = s;
      r.seg = seg;
      out.push_back(r);
    }
  };
  for (int seg = 0; seg < kNumSegs; ++seg) seg_streams_[(size_t)s * kNumSegs + seg] = 0;
  const bool merged = cfg_.merged && layer >= 0;
  for (int seg = 0; seg < kNumSegs; ++seg) {
    if (merged && seg != kSegMisc) continue;
    const int64_t bytes = seg_bytes(seg);
    if (bytes <= 0) continue;
    for (int64_t off = 0; off < bytes; off += cfg_.chunk_bytes)
      seg_streams_[(size_t)s * kNumSegs + seg] |=
          (uint8_t)(1u << copy(seg, off, std::min(cfg_.chunk_bytes, bytes - off)));
    record(seg);
  }
  if (!merged) return;
  // the matrix segments as one range from the first one's slot offset; a
  // chunk marks every segment it overlaps, and a segment's ready events are
  // recorded right after the chunk that holds its last byte
  const int64_t base = cfg_.layer_seg_off[kSegWqkv];
  int64_t end = 0;
  for (int seg = kSegWqkv; seg < kSegHead; ++seg)
    if (seg_bytes(seg) > 0) end = cfg_.layer_seg_off[seg] + seg_bytes(seg) - base;
  int next_rec = kSegWqkv;
  for (int64_t off = 0; off < end; off += cfg_.chunk_bytes) {
    const int64_t len = std::min(cfg_.chunk_bytes, end - off);
    const int st = copy(kSegWqkv, off, len);
    for (int seg = kSegWqkv; seg < kSegHead; ++seg) {
      const int64_t a = cfg_.layer_seg_off[seg] - base, b = a + seg_bytes(seg);
      if (seg_bytes(seg) > 0 && a < off + len && b > off)
        seg_streams_[(size_t)s * kNumSegs + seg] |= (uint8_t)(1u << st);
    }
    for (; next_rec < kSegHead; ++next_rec) {
      if (seg_bytes(next_rec) <= 0) continue;
      if (cfg_.layer_seg_off[next_rec] - base + seg_bytes(next_rec) > off + len) break;
      record(next_rec);
    }
  }
}

void Scheduler::issue_kv(int64_t g, const PassInfo& p, std::vector<Op>& out) {
  const int s = (int)(g % cfg_.n_slots);
  const int layer = unit_layer((int)(g % U_));
  if (layer < 0) return;
  kv_streams_[s] = 0;
  if (p.prefill) return;  // a new sequence has no prefix to load
  const int n = cfg_.n_h2d;
  for (int i = 0; i < n; ++i) {
    if (g >= cfg_.n_slots) {
      Op w = make(OpKind::Wait, kH2D0 + i);
      w.event = ev_.slot_free(s);
      w.unit = g;
      w.slot = s;
      out.push_back(w);
      Op w2 = make(OpKind::Wait, kH2D0 + i);
      w2.event = ev_.save_slot(s);
      w2.unit = g;
      w2.slot = s;
      out.push_back(w2);
    }
    Op w3 = make(OpKind::Wait, kH2D0 + i);
    w3.event = ev_.kvsave_layer(layer);
    w3.unit = g;
    w3.layer = layer;
    out.push_back(w3);
  }
  if (cfg_.poison) {
    Op po = make(OpKind::Poison, kH2D0);
    po.unit = g;
    po.slot = s;
    po.kv = true;
    out.push_back(po);
    if (n > 1) {
      Op r = make(OpKind::Record, kH2D0);
      r.event = ev_.poisoned(s);
      out.push_back(r);
      Op w = make(OpKind::Wait, kH2D1);
      w.event = ev_.poisoned(s);
      out.push_back(w);
    }
  }
  const int64_t bytes = p.pos0 * p.kv_row_bytes;
  int chunk_no = 0;
  for (int part = 0; part < 2; ++part) {
    for (int64_t off = 0; off < bytes; off += cfg_.chunk_bytes) {
      const int st = chunk_no++ % n;
      if (cfg_.delay) out.push_back(make(OpKind::Delay, kH2D0 + st));
      Op c = make(OpKind::CopyH2D, kH2D0 + st);
      c.unit = g;
      c.layer = layer;
      c.slot = s;
      c.seg = part;
      c.kv = true;
      c.off = off;
      c.bytes = std::min(cfg_.chunk_bytes, bytes - off);
      out.push_back(c);
      kv_streams_[s] |= (uint8_t)(1u << st);
    }
  }
  for (int st = 0; st < n; ++st) {
    if (!(kv_streams_[s] & (1u << st))) continue;
    Op r = make(OpKind::Record, kH2D0 + st);
    r.event = ev_.kv_ready(s, st);
    r.unit = g;
    r.slot = s;
    out.push_back(r);
  }
}

void Scheduler::wait_seg(int slot, int seg, std::vector<Op>& out) const {
  const uint8_t mask = seg_streams_[(size_t)slot * kNumSegs + seg];
  for (int st = 0; st < cfg_.n_h2d; ++st) {
    if (!(mask & (1u << st))) continue;
    Op w = make(OpKind::Wait, kCompute);
    w.event = ev_.seg_ready(slot, seg, st);
    w.slot = slot;
    w.seg = seg;
    out.push_back(w);
  }
}

void Scheduler::kernel(int k, int64_t g, int layer, int slot, std::vector<Op>& out) const {
  Op o = make(OpKind::Kernel, kCompute);
  o.kernel = k;
  o.unit = g;
  o.layer = layer;
  o.slot = slot;
  out.push_back(o);
}

void Scheduler::compute_layer(int64_t g, int j, const PassInfo& p, std::vector<Op>& out) {
  const int s = g >= 0 ? (int)(g % cfg_.n_slots) : -1;
  if (g >= 0) wait_seg(s, kSegMisc, out);
  kernel(kLn1, g, j, s, out);
  if (g >= 0) {
    wait_seg(s, kSegWqkv, out);
    wait_seg(s, kSegWqkvSm, out);
  }
  if (cfg_.kv_on_host) {
    if (!p.prefill) {
      for (int st = 0; st < cfg_.n_h2d; ++st) {
        if (!(kv_streams_[s] & (1u << st))) continue;
        Op w = make(OpKind::Wait, kCompute);
        w.event = ev_.kv_ready(s, st);
        w.slot = s;
        out.push_back(w);
      }
    }
    // the QKV projection overwrites the slot's KV buffer: its previous
    // contents must have been saved
    if (g >= cfg_.n_slots) {
      Op w = make(OpKind::Wait, kCompute);
      w.event = ev_.save_slot(s);
      w.slot = s;
      out.push_back(w);
    }
  }
  kernel(kQkv, g, j, s, out);
  if (cfg_.kv_on_host) {
    Op r = make(OpKind::Record, kCompute);
    r.event = ev_.qkv_done(s);
    r.slot = s;
    out.push_back(r);
    Op w = make(OpKind::Wait, kD2H);
    w.event = ev_.qkv_done(s);
    w.slot = s;
    out.push_back(w);
    for (int part = 0; part < 2; ++part) {
      Op c = make(OpKind::CopyD2H, kD2H);
      c.unit = g;
      c.layer = j;
      c.slot = s;
      c.seg = part;
      c.kv = true;
      c.off = p.pos0 * p.kv_row_bytes;
      c.bytes = p.T * p.kv_row_bytes;
      out.push_back(c);
    }
    Op r1 = make(OpKind::Record, kD2H);
    r1.event = ev_.kvsave_layer(j);
    r1.layer = j;
    out.push_back(r1);
    Op r2 = make(OpKind::Record, kD2H);
    r2.event = ev_.save_slot(s);
    r2.slot = s;
    out.push_back(r2);
  }
  kernel(kAttn, g, j, s, out);
  if (g >= 0) {
    wait_seg(s, kSegWo, out);
    wait_seg(s, kSegWoSm, out);
  }
  kernel(kOproj, g, j, s, out);
  kernel(kLn2, g, j, s, out);
  if (g >= 0) {
    wait_seg(s, kSegW1, out);
    wait_seg(s, kSegW1Sm, out);
  }
  kernel(kFc1, g, j, s, out);
  if (g >= 0) {
    wait_seg(s, kSegW2, out);
    wait_seg(s, kSegW2Sm, out);
  }
  kernel(kFc2, g, j, s, out);
  if (g >= 0) {
    Op r = make(OpKind::Record, kCompute);
    r.event = ev_.slot_free(s);
    r.unit = g;
    r.slot = s;
    out.push_back(r);
  }
}

void Scheduler::compute_head(int64_t g, std::vector<Op>& out) {
  const int s = g >= 0 ? (int)(g % cfg_.n_slots) : -1;
  kernel(kLnf, g, -1, s, out);
  if (g >= 0) wait_seg(s, kSegHead, out);
  kernel(kHead, g, -1, s, out);
  if (g >= 0) {
    Op r = make(OpKind::Record, kCompute);
    r.event = ev_.slot_free(s);
    r.unit = g;
    r.slot = s;
    out.push_back(r);
  }
}

void Scheduler::pass(const PassInfo& p, std::vector<Op>& out) {
  pass_base_ = g_next_;
  const int64_t pass_end = pass_base_ + U_;
  g_kv_issued_ = std::max(g_kv_issued_, pass_base_);
  const auto issue_upto = [&](int64_t last) {
    for (; g_w_issued_ <= last; ++g_w_issued_) issue_weights(g_w_issued_, out);
    if (cfg_.kv_on_host)
      for (; g_kv_issued_ <= std::min(last, pass_end - 1); ++g_kv_issued_)
        issue_kv(g_kv_issued_, p, out);
  };
  kernel(kEmbed, -1, -1, -1, out);
  int u = 0;
  for (int j = 0; j < cfg_.n_layers; ++j) {
    if (cfg_.layers_streamed) {
      const int64_t g = pass_base_ + u++;
      issue_upto(g + la_);
      compute_layer(g, j, p, out);
    } else {
      compute_layer(-1, j, p, out);
    }
  }
  if (cfg_.head_streamed) {
    const int64_t g = pass_base_ + u++;
    issue_upto(g + la_);
    compute_head(g, out);
  } else {
    compute_head(-1, out);
  }
  kernel(kArgmax, -1, -1, -1, out);
  out.push_back(make(OpKind::Readback, kCompute));
  g_next_ = pass_end;
}

std::string op_to_string(const Op& o) {
  char buf[256];
  std::snprintf(buf, sizeof buf, "%d %d %d %d %lld %d %d %d %d %lld %lld", (int)o.kind, o.stream,
                o.event, o.kernel, (long long)o.unit, o.layer, o.slot, o.seg, o.kv ? 1 : 0,
                (long long)o.off, (long long)o.bytes);
  return buf;
}

}  // namespace pipo
