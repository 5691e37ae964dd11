// C entry point returning the pipeline schedule as text (pipo_sched.h).
#include <cstring>
#include <string>
#include <vector>

#include "pipo_sched.h"
#include "schedule.h"

extern "C" int64_t pipo_sched_trace(const pipo_sched_config* c, int32_t n_passes,
                                    const int32_t* prefill, const int64_t* pos0, const int64_t* T,
                                    int64_t kv_row_bytes, char* buf, int64_t buflen) {
  if (!c || !prefill || !pos0 || !T || !buf || buflen <= 0 || n_passes < 0) return -1;
  if (c->n_layers < 1 || c->n_slots < 1 || c->n_h2d < 1 || c->n_h2d > 2 || c->chunk_bytes <= 0)
    return -1;
  if (c->kv_on_host && !c->layers_streamed) return -1;
  pipo::SchedConfig sc;
  sc.n_layers = c->n_layers;
  sc.n_slots = c->n_slots;
  sc.n_h2d = c->n_h2d;
  sc.layers_streamed = c->layers_streamed != 0;
  sc.head_streamed = c->head_streamed != 0;
  sc.kv_on_host = c->kv_on_host != 0;
  sc.chunk_bytes = c->chunk_bytes;
  for (int i = 0; i < pipo::kNumSegs; ++i) sc.layer_seg_bytes[i] = c->layer_seg_bytes[i];
  sc.layer_seg_bytes[pipo::kSegHead] = 0;
  sc.head_bytes = c->head_bytes;
  sc.merged = c->merged != 0;
  for (int i = 0; i < pipo::kNumSegs; ++i) sc.layer_seg_off[i] = c->layer_seg_off[i];
  if (sc.merged) {  // segments must follow each other in slot order without overlap
    int64_t end = sc.layer_seg_off[pipo::kSegWqkv];
    for (int i = pipo::kSegWqkv; i < pipo::kSegHead; ++i) {
      if (sc.layer_seg_bytes[i] <= 0) continue;
      if (sc.layer_seg_off[i] < end) return -1;
      end = sc.layer_seg_off[i] + sc.layer_seg_bytes[i];
    }
  }
  sc.poison = c->poison != 0;
  sc.delay = c->delay != 0;
  // no C++ exception (an exhausted heap) may leave the C entry point
  try {
    pipo::Scheduler sched(sc);
    std::string text;
    std::vector<pipo::Op> ops;
    for (int i = 0; i < n_passes; ++i) {
      pipo::PassInfo p;
      p.prefill = prefill[i] != 0;
      p.pos0 = pos0[i];
      p.T = T[i];
      p.kv_row_bytes = kv_row_bytes;
      ops.clear();
      sched.pass(p, ops);
      for (const auto& o : ops) {
        text += pipo::op_to_string(o);
        text += '\n';
      }
    }
    if ((int64_t)text.size() + 1 > buflen) return -1;
    std::memcpy(buf, text.c_str(), text.size() + 1);
    return (int64_t)text.size();
  } catch (...) {
    return -1;
  }
}
