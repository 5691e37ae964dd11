// Pipeline schedule of one pass (prefill or decode step) as an ordered list
// of stream operations.  Pure C++ (no HIP): the GPU engine executes the list
// on HIP streams; a recording executor checks its ordering on the CPU.
//
// It is PIPO's pipeline scheduling (Algorithm 1) recast for HIP streams:
//   - every streamed unit (a layer's merged tensors, or the output head)
//     goes to HBM slot g % n_slots, g counting unit instances over the
//     context's lifetime; loads run up to n_slots - 1 units ahead of the
//     unit being computed (Section 3.2.3: two or more layers resident);
//   - CallLoadData is a chain of chunk copies on the copy stream(s) that
//     first waits for the slot's previous user to finish (slot_free);
//   - SynchronizeLoadTask is a stream wait on the event recorded after the
//     last chunk of each tensor, placed right before the kernel that reads
//     it, so a layer's first GEMM never waits for its last matrix;
//   - with the KV cache in host memory, a layer's prefix is loaded into the
//     slot's KV buffer after the save of the same layer at the previous
//     token completes (Section 3.2.2: saves are checked one layer early),
//     and the new rows are saved on the device-to-host stream right after
//     the QKV projection writes them (CallStoreCache).
// Wait/Record follow CUDA/HIP event semantics: a wait refers to the most
// recent record of the event issued before it.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace pipo {

enum class OpKind : int {
  CopyH2D = 0,  // weights or KV prefix, host -> slot
  CopyD2H = 1,  // new KV rows, KV slot -> host
  Wait = 2,
  Record = 3,
  Kernel = 4,
  Delay = 5,    // host-side sleep before the next copy (debug)
  Poison = 6,   // fill a slot with NaN before it is refilled (debug)
  Readback = 7, // tokens (and logits) to the host; the host waits for it
};

enum StreamId : int { kCompute = 0, kH2D0 = 1, kH2D1 = 2, kD2H = 3, kNumStreams = 4 };

enum KernelId : int {
  kEmbed = 0, kLn1, kQkv, kAttn, kOproj, kLn2, kFc1, kFc2, kLnf, kHead, kArgmax, kNumKernels
};

// tensors of a unit, in slot order
enum SegId : int {
  kSegMisc = 0,  // LayerNorm parameters and biases, packed
  kSegWqkv, kSegWqkvSm, kSegWo, kSegWoSm, kSegW1, kSegW1Sm, kSegW2, kSegW2Sm,
  kSegHead,      // tied token table used as the output head
  kNumSegs
};

struct Op {
  OpKind kind = OpKind::Kernel;
  int stream = kCompute;
  int event = -1;
  int kernel = -1;
  int64_t unit = -1;   // unit instance g (-1: resident weights)
  int layer = -1;      // layer index, -1 for the head
  int slot = -1;       // weight/KV slot of the unit instance
  int seg = -1;        // CopyH2D of weights: segment (a merged copy names its first
                       // segment, `off` may run past its end); KV copies: 0 = K, 1 = V
  bool kv = false;     // copy of KV-cache rows
  int64_t off = 0;     // byte offset inside the segment (weights) or KV part
  int64_t bytes = 0;
};

struct SchedConfig {
  int n_layers = 0;
  int n_slots = 3;
  int n_h2d = 1;
  bool layers_streamed = true;
  bool head_streamed = true;
  bool kv_on_host = false;
  int64_t chunk_bytes = 64ll << 20;
  int64_t layer_seg_bytes[kNumSegs] = {};  // bytes of each segment of a layer unit
  int64_t head_bytes = 0;
  // merged copies: a layer's matrix segments sit in host memory at the same
  // relative offsets as in the slot (layer_seg_off), so they are copied as
  // one byte range in chunks that may span segments (fewer, larger copies;
  // Section 3.3, data merging).  The small-tensor segment is copied alone.
  bool merged = false;
  int64_t layer_seg_off[kNumSegs] = {};
  bool poison = false;
  bool delay = false;
};

struct PassInfo {
  bool prefill = true;
  int64_t pos0 = 0;   // first position this pass appends
  int64_t T = 1;      // positions this pass appends
  int64_t kv_row_bytes = 0;  // one position of one K (or V) part: b * d * 2 bytes
};

// event ids
struct Events {
  int n_slots = 0, n_layers = 0;
  int slot_free(int s) const { return s; }
  int seg_ready(int s, int seg, int st) const { return n_slots + (s * kNumSegs + seg) * 2 + st; }
  int kv_ready(int s, int st) const { return n_slots * (1 + 2 * kNumSegs) + s * 2 + st; }
  int qkv_done(int s) const { return n_slots * (3 + 2 * kNumSegs) + s; }
  int save_slot(int s) const { return n_slots * (4 + 2 * kNumSegs) + s; }
  int poisoned(int s) const { return n_slots * (5 + 2 * kNumSegs) + s; }
  int kvsave_layer(int j) const { return n_slots * (6 + 2 * kNumSegs) + j; }
  int count() const { return n_slots * (6 + 2 * kNumSegs) + n_layers; }
};

class Scheduler {
 public:
  explicit Scheduler(const SchedConfig& c);
  // append the operations of one pass to `out`
  void pass(const PassInfo& p, std::vector<Op>& out);
  const Events& events() const { return ev_; }
  int units_per_pass() const { return U_; }
  int lookahead() const { return la_; }
  // layer index of unit-in-pass u, -1 for the head
  int unit_layer(int u) const { return (cfg_.layers_streamed && u < cfg_.n_layers) ? u : -1; }

 private:
  void issue_weights(int64_t g, std::vector<Op>& out);
  void issue_kv(int64_t g, const PassInfo& p, std::vector<Op>& out);
  void wait_seg(int slot, int seg, std::vector<Op>& out) const;
  void kernel(int k, int64_t g, int layer, int slot, std::vector<Op>& out) const;
  void compute_layer(int64_t g, int layer, const PassInfo& p, std::vector<Op>& out);
  void compute_head(int64_t g, std::vector<Op>& out);

  SchedConfig cfg_;
  Events ev_;
  int U_ = 0;     // streamed units per pass
  int la_ = 0;    // lookahead in units
  int64_t g_next_ = 0;       // next unit instance to compute
  int64_t g_w_issued_ = 0;   // weights issued for instances < this
  int64_t g_kv_issued_ = 0;  // KV loads considered for instances < this
  int64_t pass_base_ = 0;    // first instance of the current pass
  // streams that carried each segment / the KV prefix of the unit in a slot
  std::vector<uint8_t> seg_streams_;  // [slot][seg] bitmask
  std::vector<uint8_t> kv_streams_;   // [slot] bitmask
};

// human-readable one-line form of an op (CPU tests)
std::string op_to_string(const Op& op);

}  // namespace pipo
