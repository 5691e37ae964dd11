// Context, executor and C ABI of the pipelined-offloading decoder
// (include/pipo.h).  The Scheduler emits each pass as a list of stream
// operations; this file owns the memory the operations refer to and runs
// them on HIP streams: hipMemcpyAsync on the copy streams (SDMA engines),
// hipStreamWaitEvent / hipEventRecord for ordering, and the HIP kernels.
//
// Memory layout
//   HBM  - weight slots: n_slots x slot_bytes; a layer unit holds its
//          segments (packed small tensors, then each matrix, INT4 codes
//          followed by their scale/min) at 4 KiB-aligned offsets;
//        - resident layers (weights_on_host = 0): n_layers units back to back;
//        - position table, final LayerNorm, token table (if resident);
//        - activations for max_batch * max_seq rows: x fp32, LN output,
//          q and attention output fp16, MLP hidden fp16, logits fp32;
//        - KV cache [n_layers][K|V][max_seq][b][d] fp16 (resident) or
//          n_slots KV buffers [K|V][max_seq][b][d] (KV in host memory).
//   host - pinned: packed small tensors per layer, copies of matrices the
//          caller did not place in pinned memory, embedding staging, token
//          readback, KV cache per layer [K|V][max_seq][b][d] (KV on host).
#include <fcntl.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cerrno>
#include <cmath>
#include <condition_variable>
#include <cstdarg>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <system_error>
#include <thread>
#include <vector>

#include "common.h"
#include "pack.h"
#include "plan.h"
#include "schedule.h"

namespace pipo {

// ---------------------------------------------------------------------------
// errors
static thread_local std::string g_err;

void set_error(const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
}
void clear_error() { g_err.clear(); }

LaunchEvents& next_launch_events() {
  static thread_local LaunchEvents ev;
  return ev;
}

// ---------------------------------------------------------------------------
// pinned host allocations made through pipo_host_alloc (base -> bytes), so a
// caller pointer can be recognised as streamable in place
static std::mutex g_pin_mu;
static std::map<uintptr_t, size_t> g_pinned;

static bool is_registered_pinned(const void* p, size_t bytes) {
  std::lock_guard<std::mutex> lk(g_pin_mu);
  const uintptr_t a = (uintptr_t)p;
  auto it = g_pinned.upper_bound(a);
  if (it == g_pinned.begin()) return false;
  --it;
  return a >= it->first && a + bytes <= it->first + it->second;
}

static void* host_alloc_pinned(size_t bytes) {
  void* p = nullptr;
  if (hipHostMalloc(&p, bytes, hipHostMallocDefault) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  try {
    std::lock_guard<std::mutex> lk(g_pin_mu);
    g_pinned[(uintptr_t)p] = bytes;
  } catch (...) {
    (void)hipHostFree(p);
    return nullptr;
  }
  return p;
}

static void host_free_pinned(void* p) {
  if (!p) return;
  {
    std::lock_guard<std::mutex> lk(g_pin_mu);
    g_pinned.erase((uintptr_t)p);
  }
  (void)hipHostFree(p);
}

// host memcpy on several threads (large weight copies at create)
static void par_memcpy(void* dst, const void* src, size_t n) {
  const size_t kMin = 64u << 20;
  const unsigned nt = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  if (n < kMin || nt == 1) {
    std::memcpy(dst, src, n);
    return;
  }
  parallel_ranges((int64_t)n, nt, [=](int64_t a, int64_t b) {
    std::memcpy((char*)dst + a, (const char*)src + a, (size_t)(b - a));
  });
}

// dst row r = table row ids[r] (row_bytes each) for r < n; large gathers on
// several threads
static void par_gather(void* dst, const void* table, const int32_t* ids, int64_t n,
                       size_t row_bytes) {
  const auto rows = [=](int64_t a, int64_t b) {
    for (int64_t r = a; r < b; ++r)
      std::memcpy((char*)dst + r * row_bytes, (const char*)table + (int64_t)ids[r] * row_bytes,
                  row_bytes);
  };
  const unsigned nt = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  if ((size_t)n * row_bytes < (64u << 20) || nt == 1) {
    rows(0, n);
    return;
  }
  parallel_ranges(n, nt, rows);
}


// Host worker threads for copies between pageable and pinned memory (the
// paper's multi-thread parallel transfer, Section 3.3): a copy is cut into
// one contiguous piece per thread; the caller runs piece 0 and waits.
class CopyPool {
 public:
  // with fewer threads than asked for when the system refuses one
  explicit CopyPool(int n) : n_(std::max(1, n)) {
    th_.reserve((size_t)n_);
    for (int i = 1; i < n_; ++i) {
      try {
        th_.emplace_back([this, i] { worker(i); });
      } catch (const std::system_error&) {
        n_ = i;
        break;
      }
    }
  }
  ~CopyPool() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto& t : th_) t.join();
  }
  void copy(void* dst, const void* src, size_t n) {
    run([=](int i) {
      const size_t per = (n + n_ - 1) / n_, a = std::min(n, i * per), b = std::min(n, a + per);
      if (b > a) std::memcpy((char*)dst + a, (const char*)src + a, b - a);
    });
  }
  void fill(void* dst, int v, size_t n) {
    run([=](int i) {
      const size_t per = (n + n_ - 1) / n_, a = std::min(n, i * per), b = std::min(n, a + per);
      if (b > a) std::memset((char*)dst + a, v, b - a);
    });
  }
  // n bytes of file `fd` at `off` into dst, one 4 KiB-aligned piece per
  // thread (direct I/O needs aligned offsets and lengths; off and n are
  // multiples of 4 KiB).  With `bounce` (pageable, 4 KiB aligned, n bytes)
  // each thread reads its piece there and copies it to dst (direct I/O
  // cannot target pinned device-mapped pages), 2 MiB at a time, so that
  // the other threads keep the disk busy while one copies and only the last
  // 2 MiB copy of each piece is left when the reads end.  False on an error
  // or a short file.
  bool pread_all(int fd, void* dst, size_t n, int64_t off, char* bounce) {
    constexpr size_t kSub = 2u << 20;
    std::atomic<bool> ok{true};
    run([&, dst, n, off, bounce](int i) {
      const size_t per = (n / n_ + 4095) / 4096 * 4096;
      const size_t a = std::min(n, i * per), b = (i == n_ - 1) ? n : std::min(n, a + per);
      char* to = bounce ? bounce : (char*)dst;
      for (size_t s = a; s < b && ok.load();) {
        const size_t e = std::min(b, s + kSub);
        for (size_t p = s; p < e && ok.load();) {
          const ssize_t r = ::pread(fd, to + p, e - p, off + (int64_t)p);
          if (r < 0 && errno == EINTR) continue;
          if (r <= 0) {
            ok = false;
            break;
          }
          p += (size_t)r;
        }
        if (bounce && ok.load()) std::memcpy((char*)dst + s, bounce + s, e - s);
        s = e;
      }
    });
    return ok.load();
  }
  // the same for writing n bytes of src at `off`
  bool pwrite_all(int fd, const void* src, size_t n, int64_t off) {
    std::atomic<bool> ok{true};
    run([&, src, n, off](int i) {
      const size_t per = (n / n_ + 4095) / 4096 * 4096;
      const size_t a = std::min(n, i * per), b = (i == n_ - 1) ? n : std::min(n, a + per);
      for (size_t p = a; p < b && ok.load();) {
        const ssize_t r = ::pwrite(fd, (const char*)src + p, b - p, off + (int64_t)p);
        if (r < 0 && errno == EINTR) continue;
        if (r <= 0) {
          ok = false;
          break;
        }
        p += (size_t)r;
      }
    });
    return ok.load();
  }

 private:
  void run(const std::function<void(int)>& fn) {
    {
      std::lock_guard<std::mutex> lk(mu_);
      job_ = fn;
      pending_ = n_ - 1;
      ++gen_;
    }
    cv_.notify_all();
    fn(0);
    std::unique_lock<std::mutex> lk(mu_);
    done_.wait(lk, [this] { return pending_ == 0; });
  }
  void worker(int i) {
    int64_t seen = 0;
    for (;;) {
      std::function<void(int)> fn;
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
        fn = job_;
      }
      fn(i);
      {
        std::lock_guard<std::mutex> lk(mu_);
        if (--pending_ == 0) done_.notify_one();
      }
    }
  }
  int n_;
  std::vector<std::thread> th_;
  std::mutex mu_;
  std::condition_variable cv_, done_;
  std::function<void(int)> job_;
  int64_t gen_ = 0;
  int pending_ = 0;
  bool stop_ = false;
};

// A ring of pinned staging buffers, each with the event of the last copy
// that used it; a D2H buffer also remembers where its data must go.
struct StagingRing {
  std::vector<char*> buf;
  std::vector<hipEvent_t> ev;
  std::vector<bool> busy;
  std::vector<char*> dst;       // D2H: pageable destination still to be filled
  std::vector<int64_t> bytes;
  int64_t buf_bytes = 0;
  int next = 0;
};

// ---------------------------------------------------------------------------
static const char* kKernelNames[kNumKernels] = {"embed", "ln1",  "qkv",  "attn", "oproj", "ln2",
                                                "fc1",   "fc2",  "lnf",  "head", "argmax"};

struct TimedRec {
  int cls;        // kernel class (kernel id * 2 + prefill), -1 for copies
  int kind;       // 0 kernel, 1 h2d copy, 2 d2h copy, 3 window begin, 4 window end
  hipEvent_t a, b;
  double bytes, flops;
};

}  // namespace pipo

using namespace pipo;

struct pipo_ctx {
  pipo_shape sh{};
  pipo_policy pol{};
  int64_t d = 0, F = 0, V = 0, L = 0, H = 0, dh = 0;
  int64_t Hkv = 0, dkv = 0;    // key/value heads and the width of a cached row
  bool llama = false;          // PIPO_FAMILY_LLAMA
  bool w4 = false;
  bool packed = false;         // layer matrices in HBM are in fragment order
  bool pack_on_copy = false;   // row-major input, converted wherever the library copies it
  int device = 0;
  hipStream_t st[kNumStreams] = {};
  std::vector<hipEvent_t> ev;
  Scheduler* sched = nullptr;
  SchedConfig scfg;
  int64_t seg_off[kNumSegs] = {};
  int64_t seg_bytes[kNumSegs] = {};
  int64_t layer_bytes = 0, head_bytes = 0, slot_bytes = 0, misc_bytes = 0;
  int64_t misc_off[kNumMisc] = {}, misc_count[kNumMisc] = {};

  // host side
  std::vector<std::vector<const void*>> layer_src;  // [L][seg] host pointer
  std::vector<std::vector<bool>> layer_copied;      // [L][seg] in the library's own region
  const void* head_src = nullptr;
  const uint16_t* tok_host = nullptr;               // for the host-side gather
  std::vector<void*> pinned;                        // library-owned pinned buffers
  int64_t pinned_bytes = 0;
  uint16_t* emb_stage = nullptr;                    // [max_batch * max_seq][d]
  int32_t* ids_stage = nullptr;                     // [max_batch * max_seq]
  int32_t* next_stage = nullptr;                    // [max_batch]
  std::vector<char*> kv_host;                       // per layer: [K|V][max_seq][b][d]
  std::vector<bool> kv_pinned;                      // per layer: pinned (else pageable, staged)
  std::vector<char*> kv_pageable;                   // pageable regions to free
  StagingRing stage_h2d, stage_d2h;
  CopyPool* pool = nullptr;
  int disk_fd = -1;                                 // disk tier: layer units in slot layout
  bool disk_direct = false;                         //   opened with O_DIRECT
  char* disk_bounce = nullptr;                      //   pageable chunk for direct I/O

  // device side
  std::vector<void*> dev;
  int64_t hbm_bytes = 0;
  char* slots = nullptr;
  char* resident = nullptr;
  uint16_t* tok_dev = nullptr;
  uint16_t* head_dev = nullptr;  // untied output head, when resident
  uint16_t* pos_dev = nullptr;
  float* rope_dev = nullptr;     // rotary (cos, sin) table [max_seq][dh/2][2]
  uint16_t* lnf_g = nullptr;
  uint16_t* lnf_b = nullptr;
  float* x = nullptr;
  uint16_t* a = nullptr;
  uint16_t* q = nullptr;
  uint16_t* o = nullptr;
  uint16_t* h = nullptr;
  uint16_t* gu = nullptr;        // SwiGLU gate and up outputs [rows][2F]
  float* logits = nullptr;
  int32_t* next_dev = nullptr;
  int32_t* ids_dev = nullptr;
  uint16_t* emb_dev = nullptr;
  float* attn_ws = nullptr;    // decode-attention split partials
  int64_t attn_ws_bytes = 0;
  float* gemm_ws = nullptr;    // GEMM K-split partials
  int64_t gemm_ws_bytes = 0;
  void* argmax_ws = nullptr;   // argmax candidates of the row partitions
  int64_t argmax_ws_bytes = 0;
  char* kv = nullptr;          // resident cache or KV slots
  bool kv4 = false;            // INT4 cache rows (PIPO_KV_INT4_G64)
  int64_t kv_row = 0;          // bytes of one cached key (value) row: 2 dkv, or 9 dkv / 16
  int64_t kv_part_bytes = 0;   // max_seq * max_batch * kv_row
  uint16_t* kst = nullptr;     // INT4 cache: fp16 staging of new (decode) or all
  uint16_t* vst = nullptr;     //   (prefill attention) key and value rows

  // sequence state
  int b = 0;
  int64_t pos = 0;   // positions held per sequence
  bool have_seq = false;
  // A pass that stopped part way leaves the schedule's view of the slots,
  // events and streams ahead of what was enqueued; the context then refuses
  // further passes (PIPO_ERR_STATE) until it is destroyed.
  bool failed = false;
  int64_t fail_after_ops = -1;   // test hook (pipo_debug_fail_pass): stop after this many ops

  // pass being executed
  PassInfo pass;
  std::vector<Op> ops;

  // statistics
  pipo_stats stats{};
  bool timestamps = false;
  bool fuse_swiglu = true;      // LLaMA decode: SwiGLU as the gate/up GEMM's epilogue
  std::vector<hipEvent_t> tpool;
  size_t tpool_used = 0;
  std::vector<TimedRec> trec;
  double kstat_ms[kNumKernels * 2] = {};
  double kstat_bytes[kNumKernels * 2] = {};
  double kstat_flops[kNumKernels * 2] = {};
  int64_t kstat_n[kNumKernels * 2] = {};
};

namespace pipo {

// ---------------------------------------------------------------------------
static pipo_status dev_alloc(pipo_ctx* c, void** p, int64_t bytes) {
  *p = nullptr;
  if (bytes <= 0) return PIPO_OK;
  if (c->pol.hbm_budget_bytes > 0 && c->hbm_bytes + bytes > c->pol.hbm_budget_bytes) {
    set_error("HBM budget exceeded: %lld + %lld > %lld bytes", (long long)c->hbm_bytes,
              (long long)bytes, (long long)c->pol.hbm_budget_bytes);
    return PIPO_ERR_OOM_DEVICE;
  }
  if (hipMalloc(p, (size_t)bytes) != hipSuccess) {
    (void)hipGetLastError();
    *p = nullptr;
    set_error("hipMalloc of %lld bytes failed", (long long)bytes);
    return PIPO_ERR_OOM_DEVICE;
  }
  c->dev.push_back(*p);
  c->hbm_bytes += bytes;
  return PIPO_OK;
}

static pipo_status pin_alloc(pipo_ctx* c, void** p, int64_t bytes) {
  *p = host_alloc_pinned((size_t)bytes);
  if (!*p) {
    set_error("pinned host allocation of %lld bytes failed", (long long)bytes);
    return PIPO_ERR_OOM_HOST;
  }
  c->pinned.push_back(*p);
  c->pinned_bytes += bytes;
  return PIPO_OK;
}

static hipEvent_t tevent(pipo_ctx* c) {
  if (c->tpool_used == c->tpool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->tpool.push_back(e);
  }
  return c->tpool[c->tpool_used++];
}

// ---------------------------------------------------------------------------
// validation

// ---------------------------------------------------------------------------
// kernels of one op
static const uint16_t* misc_ptr(const char* base, const pipo_ctx* c) {
  return reinterpret_cast<const uint16_t*>(base + c->seg_off[kSegMisc]);
}

// one small tensor of the packed block, or null where the family has none
static const uint16_t* misc_tensor(const uint16_t* misc, const pipo_ctx* c, int which) {
  return misc && c->misc_count[which] > 0 ? misc + c->misc_off[which] : nullptr;
}

static pipo_status run_kernel(pipo_ctx* c, const Op& op) {
  hipStream_t s = c->st[kCompute];
  const PassInfo& p = c->pass;
  const int64_t rows = (int64_t)c->b * p.T;
  const int64_t d = c->d, F = c->F;
  const int j = op.layer;
  // weights of the unit
  const char* base = nullptr;
  if (op.kernel != kEmbed && op.kernel != kArgmax) {
    if (op.unit >= 0) {
      base = c->slots + (int64_t)op.slot * c->slot_bytes;
    } else if (j >= 0) {
      base = c->resident + (int64_t)j * c->layer_bytes;
    } else {
      base = reinterpret_cast<const char*>(c->llama ? c->head_dev : c->tok_dev);
    }
  }
  const uint16_t* misc = base && j >= 0 ? misc_ptr(base, c) : nullptr;
  const auto small = [&](int which) { return misc_tensor(misc, c, which); };
  // KV cache of layer j (fp16 or INT4 rows, position-major)
  char *kc = nullptr, *vc = nullptr;
  if (j >= 0) {
    char* kvb = c->pol.kv_on_host ? c->kv + (int64_t)op.slot * 2 * c->kv_part_bytes
                                  : c->kv + (int64_t)j * 2 * c->kv_part_bytes;
    kc = kvb;
    vc = kvb + c->kv_part_bytes;
  }
  const auto gemm = [&](int seg, const uint16_t* X, const uint16_t* bias, int64_t M, int64_t N,
                        int64_t K, int epi, GemmArgs& ga) {
    ga.X = X;
    ga.bias = bias;
    ga.M = M;
    ga.N = N;
    ga.K = K;
    ga.packed = c->packed;
    if (c->w4) {
      ga.Wq = reinterpret_cast<const uint8_t*>(base + c->seg_off[seg]);
      ga.Wsm = reinterpret_cast<const uint16_t*>(base + c->seg_off[seg + 1]);
    } else {
      ga.W = reinterpret_cast<const uint16_t*>(base + c->seg_off[seg]);
    }
    return launch_gemm(ga, c->w4, epi, c->gemm_ws, c->gemm_ws_bytes, s);
  };
  switch (op.kernel) {
    case kEmbed: {
      if (c->pol.embed_on_host) {
        PIPO_HIP_TRY(hipMemcpyAsync(c->emb_dev, c->emb_stage, (size_t)(rows * d * 2),
                                    hipMemcpyHostToDevice, s));
        c->stats.n_copies++;
        return launch_embed(c->emb_dev, nullptr, nullptr, c->pos_dev, c->x, rows, d, p.T, p.pos0,
                            c->sh.pos_offset, s);  // pos_dev is null for LLaMA
      }
      PIPO_HIP_TRY(hipMemcpyAsync(c->ids_dev, c->ids_stage, (size_t)(rows * 4),
                                  hipMemcpyHostToDevice, s));
      c->stats.n_copies++;
      return launch_embed(nullptr, c->ids_dev, c->tok_dev, c->pos_dev, c->x, rows, d, p.T, p.pos0,
                          c->sh.pos_offset, s);
    }
    case kLn1:
      if (c->llama)
        return launch_rmsnorm(c->x, small(kLn1G), c->a, rows, d, 1, 0, c->sh.ln_eps, s);
      return launch_layernorm(c->x, small(kLn1G), small(kLn1B), c->a, rows, d, 1, 0,
                              c->sh.ln_eps, s);
    case kQkv: {
      GemmArgs ga;
      ga.q_out = c->q;
      ga.d = d;
      ga.dkv = c->dkv;
      // OPT scales q in the epilogue; LLaMA scales it with the rotation
      const float q_scale = 1.0f / std::sqrt((float)c->dh);
      ga.q_scale = c->llama ? 1.f : q_scale;
      ga.rows_per_seq = p.T;
      ga.batch = c->b;
      // fp16 cache: k and v rows go straight to the cache at pos0.  INT4
      // cache: they go to fp16 staging (position-major from the pass's first
      // position) and are quantized into the cache at pos0.
      ga.k_out = c->kv4 ? c->kst : reinterpret_cast<uint16_t*>(kc);
      ga.v_out = c->kv4 ? c->vst : reinterpret_cast<uint16_t*>(vc);
      ga.pos0 = c->kv4 ? 0 : p.pos0;
      PIPO_TRY(gemm(kSegWqkv, c->a, small(kBqkv), rows, d + 2 * c->dkv, d, EPI_QKV, ga));
      if (c->llama)  // rotary positions on q and on the new keys, where they were written
        PIPO_TRY(launch_rope(c->q, ga.k_out, c->rope_dev, rows, p.T, p.pos0, ga.pos0, c->b,
                             (int)c->H, (int)c->Hkv, (int)c->dh, q_scale, s));
      if (!c->kv4) return PIPO_OK;
      const int64_t at = p.pos0 * c->b * c->kv_row;
      PIPO_TRY(launch_kv_quant(c->kst, reinterpret_cast<uint8_t*>(kc + at), rows, c->dkv, s));
      return launch_kv_quant(c->vst, reinterpret_cast<uint8_t*>(vc + at), rows, c->dkv, s);
    }
    case kAttn:
      if (p.prefill) {
        if (!c->kv4)
          return launch_attn_prefill(c->q, reinterpret_cast<const uint16_t*>(kc),
                                     reinterpret_cast<const uint16_t*>(vc), c->o, c->b, (int)p.T,
                                     (int)c->H, (int)c->Hkv, (int)c->dh, s);
        // INT4 cache: attention reads the cache, expanded to fp16 staging
        PIPO_TRY(
            launch_kv_dequant(reinterpret_cast<const uint8_t*>(kc), c->kst, rows, c->dkv, s));
        PIPO_TRY(
            launch_kv_dequant(reinterpret_cast<const uint8_t*>(vc), c->vst, rows, c->dkv, s));
        return launch_attn_prefill(c->q, c->kst, c->vst, c->o, c->b, (int)p.T, (int)c->H,
                                   (int)c->Hkv, (int)c->dh, s);
      }
      return launch_attn_decode(c->q, kc, vc, c->o, c->b, (int)c->H, (int)c->Hkv, (int)c->dh,
                                (int)p.pos0, c->kv4, c->attn_ws, c->attn_ws_bytes, s);
    case kOproj: {
      GemmArgs ga;
      ga.out32 = c->x;
      ga.ldo = d;
      return gemm(kSegWo, c->o, small(kBo), rows, d, d, EPI_ADD_F32, ga);
    }
    case kLn2:
      if (c->llama)
        return launch_rmsnorm(c->x, small(kLn2G), c->a, rows, d, 1, 0, c->sh.ln_eps, s);
      return launch_layernorm(c->x, small(kLn2G), small(kLn2B), c->a, rows, d, 1, 0,
                              c->sh.ln_eps, s);
    case kFc1: {
      GemmArgs ga;
      if (c->llama) {  // gate and up in one GEMM, then the SwiGLU gate
        if (rows <= 16 && c->fuse_swiglu) {  // decode: the gate in the GEMM's epilogue, same values
          ga.out16 = c->h;
          ga.ldo = F;
          return gemm(kSegW1, c->a, nullptr, rows, 2 * F, d, EPI_SWIGLU, ga);
        }
        ga.out16 = c->gu;
        ga.ldo = 2 * F;
        PIPO_TRY(gemm(kSegW1, c->a, nullptr, rows, 2 * F, d, EPI_F16, ga));
        return launch_swiglu(c->gu, c->h, rows, F, s);
      }
      ga.out16 = c->h;
      ga.ldo = F;
      return gemm(kSegW1, c->a, small(kB1), rows, F, d, EPI_RELU_F16, ga);
    }
    case kFc2: {
      GemmArgs ga;
      ga.out32 = c->x;
      ga.ldo = d;
      return gemm(kSegW2, c->h, small(kB2), rows, d, F, EPI_ADD_F32, ga);
    }
    case kLnf:
      if (c->llama)
        return launch_rmsnorm(c->x, c->lnf_g, c->a, c->b, d, p.T, p.T - 1, c->sh.ln_eps, s);
      return launch_layernorm(c->x, c->lnf_g, c->lnf_b, c->a, c->b, d, p.T, p.T - 1, c->sh.ln_eps,
                              s);
    case kHead: {
      GemmArgs ga;
      ga.X = c->a;
      ga.W = reinterpret_cast<const uint16_t*>(base);  // slot offset 0, or the resident head
      ga.M = c->b;
      ga.N = c->V;
      ga.K = d;
      ga.out32 = c->logits;
      ga.ldo = c->V;
      return launch_gemm(ga, false, EPI_F32, c->gemm_ws, c->gemm_ws_bytes, s);
    }
    case kArgmax:
      return launch_argmax(c->logits, c->next_dev, c->b, c->V, c->argmax_ws, c->argmax_ws_bytes,
                           s);
    default:
      set_error("unknown kernel %d", op.kernel);
      return PIPO_ERR_ARG;
  }
}

// algorithmic bytes and flops of a kernel op (for the per-kernel roofline)
static void kernel_cost(const pipo_ctx* c, const Op& op, double* bytes, double* flops) {
  const PassInfo& p = c->pass;
  const double rows = (double)c->b * p.T, d = (double)c->d, F = (double)c->F, V = (double)c->V;
  const double dkv = (double)c->dkv;
  const auto wbytes = [&](double N, double K) { return c->w4 ? N * K / 2 + N * K / 16 : N * K * 2; };
  // weights once, X once, Y once (bias only where the family has one)
  const auto g = [&](double M, double N, double K, double out_bytes, double wb) {
    *bytes = wb + M * K * 2 + M * N * out_bytes + (c->llama ? 0 : N * 2);
    *flops = 2 * M * N * K;
  };
  *bytes = 0;
  *flops = 0;
  switch (op.kernel) {
    case kQkv: {
      const double N = d + 2 * dkv;
      g(rows, N, d, 2, wbytes(N, d));
      if (c->llama) *bytes += rows * (d + dkv) * 4;            // rotation: read and write q, k
      if (c->kv4) *bytes += 2 * rows * (dkv * 4 + c->kv_row);  // staging write, read, INT4 write
      break;
    }
    case kOproj: g(rows, d, d, 8, wbytes(d, d)); break;
    case kFc1:
      if (c->llama) {
        g(rows, 2 * F, d, 2, wbytes(2 * F, d));
        if (rows <= 16 && c->fuse_swiglu)
          *bytes -= rows * F * 2;  // SwiGLU in the epilogue: h (F columns) written instead
        else
          *bytes += rows * F * 6;  // SwiGLU: read gate and up, write h
      } else {
        g(rows, F, d, 2, wbytes(F, d));
      }
      break;
    case kFc2: g(rows, d, F, 8, wbytes(d, F)); break;
    case kHead: g(c->b, V, d, 4, V * d * 2); break;
    case kLn1:
    case kLn2: *bytes = rows * d * 6 + d * 4; *flops = rows * d * 8; break;
    case kLnf: *bytes = c->b * d * 6 + d * 4; *flops = c->b * d * 8; break;
    case kAttn:
      // K and V once (per key/value head), q and o once
      if (p.prefill) {
        *bytes = 2 * rows * (d + dkv) * 2 + (c->kv4 ? 2 * rows * (c->kv_row + dkv * 2) : 0);
        *flops = 4.0 * c->b * p.T * (p.T + 1) / 2 * d;
      } else {
        *bytes = 2.0 * c->b * (p.pos0 + 1) * c->kv_row + 2 * rows * d * 2;
        *flops = 4.0 * c->b * (p.pos0 + 1) * d;
      }
      break;
    case kEmbed: *bytes = rows * d * 8; break;
    case kArgmax: *bytes = c->b * V * 4; break;
    default: break;
  }
}

// ---------------------------------------------------------------------------
// staged copies for host KV layers in pageable memory.  They run inline in
// the executor, so every event record and wait keeps program order: a H2D
// chunk is copied by the worker threads into a free pinned buffer and DMA'd
// from there; a D2H chunk is DMA'd into a buffer and copied out to pageable
// memory when that buffer is needed again or at the end of the pass.
static pipo_status finish_d2h(pipo_ctx* c, int b) {
  StagingRing& r = c->stage_d2h;
  if (!r.busy[b]) return PIPO_OK;
  PIPO_HIP_TRY(hipEventSynchronize(r.ev[b]));
  c->pool->copy(r.dst[b], r.buf[b], (size_t)r.bytes[b]);
  r.busy[b] = false;
  return PIPO_OK;
}

static pipo_status drain_d2h(pipo_ctx* c) {
  for (size_t i = 0; i < c->stage_d2h.buf.size(); ++i) {
    const int b = (int)((c->stage_d2h.next + i) % c->stage_d2h.buf.size());  // oldest first
    PIPO_TRY(finish_d2h(c, b));
  }
  return PIPO_OK;
}

// `first` (optional) is recorded right before the first DMA, so that a
// timeline interval covers the DMA and not the host-side copy before it
static pipo_status staged_h2d(pipo_ctx* c, void* dst, const void* src, int64_t bytes,
                              hipStream_t s, hipEvent_t first) {
  StagingRing& r = c->stage_h2d;
  for (int64_t off = 0; off < bytes; off += r.buf_bytes) {
    const int64_t n = std::min(r.buf_bytes, bytes - off);
    const int b = r.next;
    r.next = (r.next + 1) % (int)r.buf.size();
    if (r.busy[b]) PIPO_HIP_TRY(hipEventSynchronize(r.ev[b]));
    c->pool->copy(r.buf[b], (const char*)src + off, (size_t)n);
    if (off == 0 && first) PIPO_HIP_TRY(hipEventRecord(first, s));
    PIPO_HIP_TRY(hipMemcpyAsync((char*)dst + off, r.buf[b], (size_t)n, hipMemcpyHostToDevice, s));
    PIPO_HIP_TRY(hipEventRecord(r.ev[b], s));
    r.busy[b] = true;
    c->stats.staged_bytes += n;
  }
  return PIPO_OK;
}

// disk tier: `bytes` of the layer file at file_off (4 KiB aligned) into HBM
// at dst through the H2D staging ring; each piece is read whole by the copy
// threads (rounded up to 4 KiB, which stays inside the file: layer units are
// 4 KiB-aligned) before its DMA is queued, so the next piece's read overlaps
// the previous piece's DMA
static pipo_status disk_h2d(pipo_ctx* c, void* dst, int64_t file_off, int64_t bytes,
                            hipStream_t s, hipEvent_t first) {
  StagingRing& r = c->stage_h2d;
  for (int64_t off = 0; off < bytes; off += r.buf_bytes) {
    const int64_t n = std::min(r.buf_bytes, bytes - off);
    const int64_t nr = align_up(n, 4096);
    const int b = r.next;
    r.next = (r.next + 1) % (int)r.buf.size();
    if (r.busy[b]) PIPO_HIP_TRY(hipEventSynchronize(r.ev[b]));
    const auto t0 = std::chrono::steady_clock::now();
    if (!c->pool->pread_all(c->disk_fd, r.buf[b], (size_t)nr, file_off + off,
                            c->disk_direct ? c->disk_bounce : nullptr)) {
      set_error("disk tier: reading %lld bytes at %lld failed: %s", (long long)nr,
                (long long)(file_off + off), std::strerror(errno));
      return PIPO_ERR_IO;
    }
    c->stats.disk_read_ms +=
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    c->stats.disk_read_bytes += nr;
    if (off == 0 && first) PIPO_HIP_TRY(hipEventRecord(first, s));
    PIPO_HIP_TRY(hipMemcpyAsync((char*)dst + off, r.buf[b], (size_t)n, hipMemcpyHostToDevice, s));
    PIPO_HIP_TRY(hipEventRecord(r.ev[b], s));
    r.busy[b] = true;
    c->stats.staged_bytes += n;
  }
  return PIPO_OK;
}

static pipo_status staged_d2h(pipo_ctx* c, void* dst, const void* src, int64_t bytes,
                              hipStream_t s, hipEvent_t first) {
  StagingRing& r = c->stage_d2h;
  for (int64_t off = 0; off < bytes; off += r.buf_bytes) {
    const int64_t n = std::min(r.buf_bytes, bytes - off);
    const int b = r.next;
    r.next = (r.next + 1) % (int)r.buf.size();
    PIPO_TRY(finish_d2h(c, b));
    if (off == 0 && first) PIPO_HIP_TRY(hipEventRecord(first, s));
    PIPO_HIP_TRY(hipMemcpyAsync(r.buf[b], (const char*)src + off, (size_t)n, hipMemcpyDeviceToHost,
                                s));
    PIPO_HIP_TRY(hipEventRecord(r.ev[b], s));
    r.busy[b] = true;
    r.dst[b] = (char*)dst + off;
    r.bytes[b] = n;
    c->stats.staged_bytes += n;
  }
  return PIPO_OK;
}

static void delay_cb(void* arg) {
  const int64_t us = (int64_t)(intptr_t)arg;
  std::this_thread::sleep_for(std::chrono::microseconds(us));
}

static pipo_status exec_op(pipo_ctx* c, const Op& op) {
  hipStream_t s = c->st[op.stream];
  switch (op.kind) {
    case OpKind::Wait:
      PIPO_HIP_TRY(hipStreamWaitEvent(s, c->ev[op.event], 0));
      return PIPO_OK;
    case OpKind::Record:
      PIPO_HIP_TRY(hipEventRecord(c->ev[op.event], s));
      return PIPO_OK;
    case OpKind::Delay:
      PIPO_HIP_TRY(hipLaunchHostFunc(s, delay_cb, (void*)(intptr_t)c->pol.copy_delay_us));
      return PIPO_OK;
    case OpKind::Poison: {
      if (op.kv)
        return launch_fill_u16(reinterpret_cast<uint16_t*>(c->kv + (int64_t)op.slot * 2 * c->kv_part_bytes),
                               0x7E00, c->kv_part_bytes, s);
      return launch_fill_u16(reinterpret_cast<uint16_t*>(c->slots + (int64_t)op.slot * c->slot_bytes),
                             0x7E00, c->slot_bytes / 2, s);
    }
    case OpKind::CopyH2D:
    case OpKind::CopyD2H: {
      void* dst;
      const void* src;
      const bool h2d = op.kind == OpKind::CopyH2D;
      if (op.kv) {
        // host cache of the layer: [K|V][max_seq][b] rows for the current batch b
        const int64_t host_off = (int64_t)op.seg * c->pol.max_seq * c->b * c->kv_row;
        char* hptr = c->kv_host[op.layer] + host_off + op.off;
        char* dptr = c->kv + (int64_t)op.slot * 2 * c->kv_part_bytes + op.seg * c->kv_part_bytes + op.off;
        dst = h2d ? (void*)dptr : (void*)hptr;
        src = h2d ? (const void*)hptr : (const void*)dptr;
      } else {
        const char* hbase = reinterpret_cast<const char*>(
            op.layer >= 0 ? c->layer_src[op.layer][op.seg] : c->head_src);
        src = hbase + op.off;
        dst = c->slots + (int64_t)op.slot * c->slot_bytes +
              (op.layer >= 0 ? c->seg_off[op.seg] : 0) + op.off;
      }
      hipEvent_t e0 = nullptr, e1 = nullptr;
      if (c->timestamps) {
        e0 = tevent(c);
        e1 = tevent(c);
      }
      if (!op.kv && op.layer >= 0 && c->disk_fd >= 0) {
        const int64_t file_off = (int64_t)op.layer * c->layer_bytes + c->seg_off[op.seg] + op.off;
        PIPO_TRY(disk_h2d(c, dst, file_off, op.bytes, s, e0));
      } else if (op.kv && !c->kv_pinned[op.layer]) {
        PIPO_TRY(h2d ? staged_h2d(c, dst, src, op.bytes, s, e0)
                     : staged_d2h(c, dst, src, op.bytes, s, e0));
      } else {
        if (e0) PIPO_HIP_TRY(hipEventRecord(e0, s));
        PIPO_HIP_TRY(hipMemcpyAsync(dst, src, (size_t)op.bytes,
                                    h2d ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost, s));
      }
      if (c->timestamps) {
        PIPO_HIP_TRY(hipEventRecord(e1, s));
        c->trec.push_back(TimedRec{-1, h2d ? 1 : 2, e0, e1, (double)op.bytes, 0});
      }
      c->stats.n_copies++;
      if (h2d) {
        c->stats.h2d_bytes += op.bytes;
        (op.kv ? c->stats.h2d_kv_bytes : c->stats.h2d_weight_bytes) += op.bytes;
      } else {
        c->stats.d2h_bytes += op.bytes;
      }
      return PIPO_OK;
    }
    case OpKind::Kernel: {
      hipEvent_t e0 = nullptr, e1 = nullptr;
      if (c->timestamps) {
        e0 = tevent(c);
        e1 = tevent(c);
        next_launch_events() = LaunchEvents{e0, e1};
      }
      const pipo_status ks = run_kernel(c, op);
      const bool unused = next_launch_events().start != nullptr;
      next_launch_events() = LaunchEvents{};
      PIPO_TRY(ks);
      c->stats.n_kernels++;
      if (c->timestamps && !unused) {
        double by, fl;
        kernel_cost(c, op, &by, &fl);
        c->trec.push_back(TimedRec{op.kernel * 2 + (c->pass.prefill ? 1 : 0), 0, e0, e1, by, fl});
      }
      return PIPO_OK;
    }
    case OpKind::Readback: {
      PIPO_HIP_TRY(hipMemcpyAsync(c->next_stage, c->next_dev, (size_t)c->b * 4,
                                  hipMemcpyDeviceToHost, s));
      c->stats.d2h_bytes += (int64_t)c->b * 4;
      c->stats.n_copies++;
      return PIPO_OK;
    }
  }
  set_error("unknown op kind");
  return PIPO_ERR_ARG;
}

static pipo_status run_pass_ops(pipo_ctx* c, float* logits_out, int32_t* next_out, bool decode) {
  c->ops.clear();
  c->sched->pass(c->pass, c->ops);
  hipEvent_t w0 = nullptr, w1 = nullptr;
  if (c->timestamps && decode) {
    w0 = tevent(c);
    PIPO_HIP_TRY(hipEventRecord(w0, c->st[kCompute]));
  }
  for (size_t i = 0; i < c->ops.size(); ++i) {
    if (c->fail_after_ops >= 0 && (int64_t)i == c->fail_after_ops) {
      c->fail_after_ops = -1;
      set_error("pass stopped after %lld of %lld ops (pipo_debug_fail_pass)", (long long)i,
                (long long)c->ops.size());
      return PIPO_ERR_HIP;
    }
    PIPO_TRY(exec_op(c, c->ops[i]));
  }
  if (c->timestamps && decode) {
    w1 = tevent(c);
    PIPO_HIP_TRY(hipEventRecord(w1, c->st[kCompute]));
    c->trec.push_back(TimedRec{-1, 3, w0, w1, 0, 0});
  }
  PIPO_HIP_TRY(hipStreamSynchronize(c->st[kCompute]));
  if (c->pool) PIPO_TRY(drain_d2h(c));   // the pass's KV saves reach pageable memory
  std::memcpy(next_out, c->next_stage, (size_t)c->b * 4);
  if (logits_out) {
    PIPO_HIP_TRY(hipMemcpy(logits_out, c->logits, (size_t)c->b * c->V * 4, hipMemcpyDeviceToHost));
    c->stats.d2h_bytes += (int64_t)c->b * c->V * 4;
  }
  return PIPO_OK;
}

// A pass that fails (or throws) after the schedule planned it: wait for
// everything already enqueued on the context's streams (and the host copy
// threads), so no copy or kernel is left running against memory the caller
// may free, then refuse further passes.
static pipo_status run_pass(pipo_ctx* c, float* logits_out, int32_t* next_out, bool decode) {
  pipo_status s = PIPO_ERR_OOM_HOST;
  std::string msg;
  try {
    s = run_pass_ops(c, logits_out, next_out, decode);
  } catch (...) {
    s = guarded([]() -> pipo_status { throw; });
  }
  if (s == PIPO_OK) return s;
  msg = pipo_last_error();
  for (int i = 0; i < kNumStreams; ++i)
    if (c->st[i]) (void)hipStreamSynchronize(c->st[i]);
  (void)hipGetLastError();
  c->failed = true;
  c->have_seq = false;
  set_error("%s (the context can no longer run passes; destroy it)", msg.c_str());
  return s;
}

// ---------------------------------------------------------------------------
static void destroy_ctx(pipo_ctx* c) {
  if (!c) return;
  (void)hipSetDevice(c->device);
  for (int i = 0; i < kNumStreams; ++i)
    if (c->st[i]) (void)hipStreamSynchronize(c->st[i]);
  for (StagingRing* r : {&c->stage_h2d, &c->stage_d2h})
    for (auto e : r->ev) (void)hipEventDestroy(e);
  delete c->pool;
  if (c->disk_fd >= 0) ::close(c->disk_fd);  // the file was unlinked when it was created
  std::free(c->disk_bounce);
  for (char* p : c->kv_pageable) std::free(p);
  for (auto e : c->ev) (void)hipEventDestroy(e);
  for (auto e : c->tpool) (void)hipEventDestroy(e);
  for (int i = 0; i < kNumStreams; ++i)
    if (c->st[i]) (void)hipStreamDestroy(c->st[i]);
  for (void* p : c->dev) (void)hipFree(p);
  for (void* p : c->pinned) host_free_pinned(p);
  delete c->sched;
  delete c;
}

// (N, K) of the matrix a segment belongs to
static void seg_matrix(const pipo_ctx* c, int sg, int64_t* N, int64_t* K) {
  const int m = (sg - kSegWqkv) / 2;
  const int64_t rows[4] = {qkv_rows(c->sh), c->d, fc1_rows(c->sh), c->d};
  const int64_t cols[4] = {c->d, c->d, c->d, c->F};
  *N = rows[m];
  *K = cols[m];
}

// a matrix segment converted from row-major to fragment order into dst
static void pack_segment(const pipo_ctx* c, int sg, const void* src, void* dst) {
  int64_t N, K;
  seg_matrix(c, sg, &N, &K);
  if (!c->w4)
    pack_f16(static_cast<const uint16_t*>(src), static_cast<uint16_t*>(dst), N, K);
  else if ((sg - kSegWqkv) % 2 == 0)
    pack_w4_codes(static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), N, K);
  else
    pack_w4_scale_min(static_cast<const uint16_t*>(src), static_cast<uint16_t*>(dst), N, K);
}

// the bytes of segment sg of layer j as they go to HBM (converted into tmp
// when the library converts what it copies)
static const char* seg_bytes_for_device(const pipo_ctx* c, int64_t j, int sg,
                                        std::vector<char>& tmp) {
  const char* src = static_cast<const char*>(c->layer_src[j][sg]);
  if (!c->pack_on_copy || sg == kSegMisc || src == nullptr || c->layer_copied[j][sg]) return src;
  tmp.resize((size_t)c->seg_bytes[sg]);
  pack_segment(c, sg, src, tmp.data());
  return tmp.data();
}

// The disk tier's file: every layer unit in slot layout (small tensors,
// then the matrices at their 4 KiB-aligned offsets, zero padding), layer j
// at j * layer_bytes.  Created in disk_dir and unlinked at once, so it
// disappears with the context (or the process); opened for direct I/O
// where the file system allows it, so that reads come from the device.
static pipo_status write_disk_tier(pipo_ctx* c) {
  const std::string dir = c->pol.disk_dir && c->pol.disk_dir[0] ? c->pol.disk_dir : ".";
  std::string path = dir + "/pipo_weights_XXXXXX";
  int fd = ::mkstemp(&path[0]);
  if (fd < 0) {
    set_error("disk tier: cannot create a file in %s: %s", dir.c_str(), std::strerror(errno));
    return PIPO_ERR_IO;
  }
  const int fd_direct = ::open(path.c_str(), O_RDWR | O_DIRECT);
  if (fd_direct >= 0) {
    ::close(fd);
    fd = fd_direct;
    c->disk_direct = true;
  }
  ::unlink(path.c_str());
  c->disk_fd = fd;
  c->disk_bounce = static_cast<char*>(std::aligned_alloc(4096, (size_t)c->pol.chunk_bytes));
  if (!c->disk_bounce) {
    set_error("disk tier: host allocation of %lld bytes failed", (long long)c->pol.chunk_bytes);
    return PIPO_ERR_OOM_HOST;
  }
  const int64_t total = c->L * c->layer_bytes;
  const int rc = ::posix_fallocate(fd, 0, (off_t)total);
  if (rc != 0) {
    set_error("disk tier: cannot reserve %lld bytes in %s: %s", (long long)total, dir.c_str(),
              std::strerror(rc));
    return PIPO_ERR_IO;
  }
  char* buf = c->disk_bounce;  // pageable: direct I/O cannot use pinned pages
  const int64_t piece = c->pol.chunk_bytes;
  std::vector<std::vector<char>> tmp((size_t)kNumSegs);
  for (int64_t j = 0; j < c->L; ++j) {
    const char* seg_src[kNumSegs] = {};
    for (int sg = 0; sg < kNumSegs; ++sg)
      if (sg != kSegHead && c->seg_bytes[sg] > 0)
        seg_src[sg] = seg_bytes_for_device(c, j, sg, tmp[(size_t)sg]);
    for (int64_t o = 0; o < c->layer_bytes; o += piece) {
      const int64_t n = std::min(piece, c->layer_bytes - o);
      int64_t cursor = o;  // [o, cursor) is filled
      for (int sg = 0; sg < kNumSegs; ++sg) {
        if (sg == kSegHead || c->seg_bytes[sg] == 0) continue;
        const int64_t lo = std::max(o, c->seg_off[sg]);
        const int64_t hi = std::min(o + n, c->seg_off[sg] + c->seg_bytes[sg]);
        if (lo >= hi) continue;
        if (lo > cursor) std::memset(buf + (cursor - o), 0, (size_t)(lo - cursor));
        c->pool->copy(buf + (lo - o), seg_src[sg] + (lo - c->seg_off[sg]), (size_t)(hi - lo));
        cursor = hi;
      }
      if (cursor < o + n) std::memset(buf + (cursor - o), 0, (size_t)(o + n - cursor));
      if (!c->pool->pwrite_all(fd, buf, (size_t)n, j * c->layer_bytes + o)) {
        set_error("disk tier: writing %lld bytes to %s failed: %s", (long long)n, dir.c_str(),
                  std::strerror(errno));
        return PIPO_ERR_IO;
      }
    }
    for (int sg = 0; sg < kNumSegs; ++sg)
      if (sg != kSegMisc) c->layer_src[j][sg] = nullptr;  // caller memory: not kept
  }
  return PIPO_OK;
}

static pipo_status create_ctx(const pipo_shape* shape, const pipo_host_weights* w,
                              const pipo_policy* policy, pipo_ctx* c) {
  PIPO_TRY(check_shape(shape));
  const bool llama = is_llama(*shape);
  if (!w || !policy || !w->tok_emb || !w->lnf_g || !w->layers ||
      (llama ? !w->lm_head : (!w->pos_emb || !w->lnf_b))) {
    set_error("weights or policy incomplete");
    return PIPO_ERR_ARG;
  }
  c->sh = *shape;
  c->pol = *policy;
  pipo_policy& pol = c->pol;
  PIPO_TRY(normalize_policy(shape, &pol));
  c->kv4 = pol.kv_fmt == PIPO_KV_INT4_G64;
  c->w4 = pol.wfmt == PIPO_W_INT4_G64;
  c->d = shape->d_model;
  c->F = shape->d_ffn;
  c->V = shape->vocab;
  c->L = shape->n_layers;
  c->H = shape->n_heads;
  c->dh = c->d / c->H;
  c->Hkv = kv_heads(*shape);
  c->dkv = kv_width(*shape);
  c->llama = llama;
  c->timestamps = (pol.debug_flags & PIPO_DBG_TIMESTAMPS) != 0;
  c->fuse_swiglu = (pol.debug_flags & PIPO_DBG_UNFUSED) == 0;
  PIPO_HIP_TRY(hipGetDevice(&c->device));
  const int64_t d = c->d, F = c->F, V = c->V, L = c->L;

  // unit layout and device allocations (plan.h: the same sizes pipo_plan_policy reports)
  const UnitLayout ul = unit_layout(*shape, c->w4);
  const HbmPlan hp = hbm_plan(*shape, pol);
  for (int sg = 0; sg < kNumSegs; ++sg) {
    c->seg_bytes[sg] = ul.seg_bytes[sg];
    c->seg_off[sg] = ul.seg_off[sg];
  }
  c->misc_bytes = ul.misc_bytes;
  for (int i = 0; i < kNumMisc; ++i) {
    c->misc_off[i] = ul.misc_off[i];
    c->misc_count[i] = ul.misc_count[i];
  }
  c->layer_bytes = ul.layer_bytes;
  c->head_bytes = ul.head_bytes;
  c->slot_bytes = hp.slot_bytes;

  // host sources: small tensors packed per layer; matrices in place when
  // they sit in pipo_host_alloc memory, else copied into a merged pinned
  // region per layer (data merging, Section 3.3)
  // layer matrices that stream from host memory must be pinned; with the
  // disk tier they are only read once, to write the file
  const bool need_host = pol.weights_on_host != 0 && !pol.weights_on_disk;
  c->layer_src.assign((size_t)L, std::vector<const void*>(kNumSegs, nullptr));
  c->layer_copied.assign((size_t)L, std::vector<bool>(kNumSegs, false));
  const auto layer_mats = [&](int64_t j, const void* (&mats)[8]) {
    const pipo_layer_host& lw = w->layers[j];
    if (c->w4) {
      const pipo_q4* q4[4] = {&lw.qqkv, &lw.qo, &lw.q1, &lw.q2};
      for (int i = 0; i < 4; ++i) {
        mats[2 * i] = q4[i]->q;
        mats[2 * i + 1] = q4[i]->scale_min;
      }
    } else {
      const uint16_t* m16[4] = {lw.wqkv, lw.wo, lw.w1, lw.w2};
      for (int i = 0; i < 4; ++i) {
        mats[2 * i] = m16[i];
        mats[2 * i + 1] = nullptr;
      }
    }
  };
  // Layout: fragment order unless row-major matrices would be streamed in
  // place from pinned caller memory (then everything stays row-major)
  if (w->layout != PIPO_LAYOUT_ROW_MAJOR && w->layout != PIPO_LAYOUT_FRAGMENT) {
    set_error("unknown weight layout %d", w->layout);
    return PIPO_ERR_ARG;
  }
  bool in_place_row_major = false;
  if (w->layout == PIPO_LAYOUT_ROW_MAJOR && need_host)
    for (int64_t j = 0; j < L && !in_place_row_major; ++j) {
      const void* mats[8];
      layer_mats(j, mats);
      for (int i = 0; i < 8; ++i)
        if (c->seg_bytes[kSegWqkv + i] > 0 && mats[i] &&
            is_registered_pinned(mats[i], (size_t)c->seg_bytes[kSegWqkv + i]))
          in_place_row_major = true;
    }
  c->packed = w->layout == PIPO_LAYOUT_FRAGMENT || !in_place_row_major;
  c->pack_on_copy = c->packed && w->layout == PIPO_LAYOUT_ROW_MAJOR;
  // every layer's small tensors, back to back; a layer's copy takes
  // seg_bytes[kSegMisc] >= misc_bytes bytes (the minimum DMA copy), so the
  // region ends with that much zero padding after the last layer
  void* misc_all = nullptr;
  const int64_t misc_region = L * c->misc_bytes + (c->seg_bytes[kSegMisc] - c->misc_bytes);
  PIPO_TRY(pin_alloc(c, &misc_all, misc_region));
  std::memset(misc_all, 0, (size_t)misc_region);
  for (int64_t j = 0; j < L; ++j) {
    const pipo_layer_host& lw = w->layers[j];
    const uint16_t* small[kNumMisc] = {lw.ln1_g, lw.ln1_b, lw.bqkv, lw.bo,
                                       lw.ln2_g, lw.ln2_b, lw.b1,   lw.b2};
    uint16_t* dst = reinterpret_cast<uint16_t*>((char*)misc_all + j * c->misc_bytes);
    for (int i = 0; i < kNumMisc; ++i) {
      if (c->misc_count[i] == 0) continue;  // not part of this family
      if (!small[i]) {
        set_error("layer %lld: small tensor %d is NULL", (long long)j, i);
        return PIPO_ERR_ARG;
      }
      std::memcpy(dst + c->misc_off[i], small[i], (size_t)c->misc_count[i] * 2);
    }
    c->layer_src[j][kSegMisc] = (char*)misc_all + j * c->misc_bytes;
    const void* mats[8];
    layer_mats(j, mats);
    int64_t copy_bytes = 0;
    for (int i = 0; i < 8; ++i) {
      const int sg = kSegWqkv + i;
      if (c->seg_bytes[sg] == 0) continue;
      if (!mats[i]) {
        set_error("layer %lld: matrix segment %d is NULL", (long long)j, sg);
        return PIPO_ERR_ARG;
      }
      c->layer_src[j][sg] = mats[i];
      if (need_host && !is_registered_pinned(mats[i], (size_t)c->seg_bytes[sg]))
        copy_bytes = align_up(copy_bytes + c->seg_bytes[sg], 4096);
    }
    if (copy_bytes > 0) {
      void* merged = nullptr;
      PIPO_TRY(pin_alloc(c, &merged, copy_bytes));
      int64_t o2 = 0;
      for (int i = 0; i < 8; ++i) {
        const int sg = kSegWqkv + i;
        if (c->seg_bytes[sg] == 0 || is_registered_pinned(mats[i], (size_t)c->seg_bytes[sg]))
          continue;
        if (c->pack_on_copy)
          pack_segment(c, sg, mats[i], (char*)merged + o2);
        else
          par_memcpy((char*)merged + o2, mats[i], (size_t)c->seg_bytes[sg]);
        c->layer_src[j][sg] = (char*)merged + o2;
        c->layer_copied[j][sg] = true;  // already in the device layout
        o2 = align_up(o2 + c->seg_bytes[sg], 4096);
      }
    }
  }
  c->tok_host = w->tok_emb;
  const uint16_t* head_host = llama ? w->lm_head : w->tok_emb;  // OPT ties the head
  c->head_src = head_host;
  if (pol.embed_on_host && !is_registered_pinned(head_host, (size_t)c->head_bytes)) {
    void* t = nullptr;
    PIPO_TRY(pin_alloc(c, &t, c->head_bytes));
    par_memcpy(t, head_host, (size_t)c->head_bytes);
    c->head_src = t;
  }

  // streams (default priority) and ordering events
  for (int i = 0; i < kNumStreams; ++i) PIPO_HIP_TRY(hipStreamCreateWithFlags(&c->st[i], hipStreamNonBlocking));
  c->scfg.n_layers = (int)L;
  c->scfg.n_slots = pol.n_weight_slots;
  c->scfg.n_h2d = pol.n_h2d_streams;
  c->scfg.layers_streamed = pol.weights_on_host != 0;
  c->scfg.head_streamed = pol.embed_on_host != 0;
  c->scfg.kv_on_host = pol.kv_on_host != 0;
  c->scfg.chunk_bytes = pol.chunk_bytes;
  for (int sg = 0; sg < kNumSegs; ++sg) {
    c->scfg.layer_seg_bytes[sg] = c->seg_bytes[sg];
    c->scfg.layer_seg_off[sg] = c->seg_off[sg];
  }
  c->scfg.layer_seg_bytes[kSegHead] = 0;
  // merged copies when every layer's matrices sit in one pinned allocation
  // at the slot's relative offsets (caller regions from pipo_host_alloc laid
  // out that way, or the library's merged regions)
  if (pol.weights_on_disk && !(pol.debug_flags & PIPO_DBG_SEGMENT_COPIES)) {
    c->scfg.merged = true;  // the file holds every unit in slot layout
  } else if (pol.weights_on_host && !(pol.debug_flags & PIPO_DBG_SEGMENT_COPIES)) {
    int last = kSegWqkv;
    for (int sg = kSegWqkv; sg < kSegHead; ++sg)
      if (c->seg_bytes[sg] > 0) last = sg;
    const int64_t span = c->seg_off[last] + c->seg_bytes[last] - c->seg_off[kSegWqkv];
    bool merged = true;
    for (int64_t j = 0; j < L && merged; ++j) {
      const char* base = static_cast<const char*>(c->layer_src[j][kSegWqkv]);
      for (int sg = kSegWqkv; sg < kSegHead; ++sg)
        if (c->seg_bytes[sg] > 0 && static_cast<const char*>(c->layer_src[j][sg]) - base !=
                                        c->seg_off[sg] - c->seg_off[kSegWqkv])
          merged = false;
      if (merged && !is_registered_pinned(base, (size_t)span)) merged = false;
    }
    c->scfg.merged = merged;
  }
  c->scfg.head_bytes = c->head_bytes;
  c->scfg.poison = (pol.debug_flags & PIPO_DBG_POISON_SLOTS) != 0;
  c->scfg.delay = (pol.debug_flags & PIPO_DBG_COPY_DELAY) != 0;
  c->sched = new Scheduler(c->scfg);
  c->ev.resize((size_t)c->sched->events().count(), nullptr);
  for (auto& e : c->ev) PIPO_HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));

  // HBM
  const int64_t rows = (int64_t)pol.max_batch * pol.max_seq;
  void* p = nullptr;
  if (hp.slots > 0) {
    PIPO_TRY(dev_alloc(c, &p, hp.slots));
    c->slots = (char*)p;
  }
  if (!pol.weights_on_host) {
    PIPO_TRY(dev_alloc(c, &p, hp.resident));
    c->resident = (char*)p;
    std::vector<char> tmp;
    for (int64_t j = 0; j < L; ++j)
      for (int sg = 0; sg < kNumSegs; ++sg)
        if (c->seg_bytes[sg] > 0 && sg != kSegHead)
          PIPO_HIP_TRY(hipMemcpy(c->resident + j * c->layer_bytes + c->seg_off[sg],
                                 seg_bytes_for_device(c, j, sg, tmp), (size_t)c->seg_bytes[sg],
                                 hipMemcpyHostToDevice));
  }
  if (!pol.embed_on_host) {
    PIPO_TRY(dev_alloc(c, &p, hp.tok));
    c->tok_dev = (uint16_t*)p;
    PIPO_HIP_TRY(hipMemcpy(c->tok_dev, w->tok_emb, (size_t)c->head_bytes, hipMemcpyHostToDevice));
  }
  if (hp.head > 0) {
    PIPO_TRY(dev_alloc(c, &p, hp.head));
    c->head_dev = (uint16_t*)p;
    PIPO_HIP_TRY(
        hipMemcpy(c->head_dev, w->lm_head, (size_t)c->head_bytes, hipMemcpyHostToDevice));
  }
  if (hp.pos > 0) {
    PIPO_TRY(dev_alloc(c, &p, hp.pos));
    c->pos_dev = (uint16_t*)p;
    PIPO_HIP_TRY(hipMemcpy(c->pos_dev, w->pos_emb, (size_t)hp.pos, hipMemcpyHostToDevice));
  }
  if (hp.rope > 0) {
    PIPO_TRY(dev_alloc(c, &p, hp.rope));
    c->rope_dev = (float*)p;
    std::vector<float> table((size_t)(hp.rope / 4));
    rope_table(*shape, pol.max_seq, table.data());
    PIPO_HIP_TRY(hipMemcpy(c->rope_dev, table.data(), (size_t)hp.rope, hipMemcpyHostToDevice));
  }
  PIPO_TRY(dev_alloc(c, &p, hp.lnf));
  c->lnf_g = (uint16_t*)p;
  c->lnf_b = c->lnf_g + d;
  PIPO_HIP_TRY(hipMemcpy(c->lnf_g, w->lnf_g, (size_t)d * 2, hipMemcpyHostToDevice));
  if (!llama)
    PIPO_HIP_TRY(hipMemcpy(c->lnf_b, w->lnf_b, (size_t)d * 2, hipMemcpyHostToDevice));
  PIPO_TRY(dev_alloc(c, &p, hp.x));
  c->x = (float*)p;
  PIPO_TRY(dev_alloc(c, &p, hp.a));
  c->a = (uint16_t*)p;
  PIPO_TRY(dev_alloc(c, &p, hp.q));
  c->q = (uint16_t*)p;
  PIPO_TRY(dev_alloc(c, &p, hp.o));
  c->o = (uint16_t*)p;
  PIPO_TRY(dev_alloc(c, &p, hp.h));
  c->h = (uint16_t*)p;
  if (hp.gu > 0) {
    PIPO_TRY(dev_alloc(c, &p, hp.gu));
    c->gu = (uint16_t*)p;
  }
  PIPO_TRY(dev_alloc(c, &p, hp.logits));
  c->logits = (float*)p;
  PIPO_TRY(dev_alloc(c, &p, hp.next));
  c->next_dev = (int32_t*)p;
  PIPO_TRY(dev_alloc(c, &p, hp.ids));
  c->ids_dev = (int32_t*)p;
  if (hp.emb > 0) {
    PIPO_TRY(dev_alloc(c, &p, hp.emb));
    c->emb_dev = (uint16_t*)p;
  }
  c->attn_ws_bytes = hp.attn_ws;
  PIPO_TRY(dev_alloc(c, &p, c->attn_ws_bytes));
  c->attn_ws = (float*)p;
  // GEMM rows: b (decode) or b * P (prefill), at most max_batch * max_seq
  c->gemm_ws_bytes = hp.gemm_ws;
  if (c->gemm_ws_bytes > 0) {
    PIPO_TRY(dev_alloc(c, &p, c->gemm_ws_bytes));
    c->gemm_ws = (float*)p;
  }
  c->argmax_ws_bytes = hp.argmax_ws;
  if (c->argmax_ws_bytes > 0) PIPO_TRY(dev_alloc(c, &c->argmax_ws, c->argmax_ws_bytes));
  c->kv_row = hp.kv_row;
  c->kv_part_bytes = hp.kv_part;
  if (hp.kstage > 0) {
    PIPO_TRY(dev_alloc(c, &p, hp.kstage));
    c->kst = (uint16_t*)p;
    PIPO_TRY(dev_alloc(c, &p, hp.kstage));
    c->vst = (uint16_t*)p;
  }
  PIPO_TRY(dev_alloc(c, &p, hp.kv));
  c->kv = (char*)p;

  // pinned staging
  if (pol.embed_on_host) {
    PIPO_TRY(pin_alloc(c, &p, rows * d * 2));
    c->emb_stage = (uint16_t*)p;
  }
  PIPO_TRY(pin_alloc(c, &p, rows * 4));
  c->ids_stage = (int32_t*)p;
  PIPO_TRY(pin_alloc(c, &p, (int64_t)pol.max_batch * 4));
  c->next_stage = (int32_t*)p;
  if (pol.kv_on_host || pol.weights_on_disk) {
    // pinned staging rings (disk reads and pageable KV layers) and the copy threads
    c->pool = new CopyPool(pol.copy_threads > 0 ? pol.copy_threads : 8);
    const int64_t buf_bytes = pol.chunk_bytes;
    for (auto [ring, n] :
         {std::pair<StagingRing*, int>{&c->stage_h2d, kStageH2DBufs},
          std::pair<StagingRing*, int>{&c->stage_d2h, pol.kv_on_host ? kStageD2HBufs : 0}}) {
      ring->buf_bytes = buf_bytes;
      ring->buf.assign((size_t)n, nullptr);
      ring->ev.assign((size_t)n, nullptr);
      ring->busy.assign((size_t)n, false);
      ring->dst.assign((size_t)n, nullptr);
      ring->bytes.assign((size_t)n, 0);
      for (int i = 0; i < n; ++i) {
        PIPO_TRY(pin_alloc(c, &p, buf_bytes));
        ring->buf[(size_t)i] = (char*)p;
        PIPO_HIP_TRY(hipEventCreateWithFlags(&ring->ev[(size_t)i], hipEventDisableTiming));
      }
    }
  }
  if (pol.weights_on_disk) PIPO_TRY(write_disk_tier(c));
  if (pol.kv_on_host) {
    // One region per layer.  Layers are pinned while the budget and the
    // system allow (the copy engines stream those directly); the rest live
    // in pageable memory and go through the pinned staging rings, with 1 GiB
    // of pinned memory held back meanwhile so that the KV layers do not take
    // the last of what the system grants.
    const int64_t per_layer = align_up(2 * c->kv_part_bytes, 4096);
    const bool force_pageable = (pol.debug_flags & PIPO_DBG_KV_PAGEABLE) != 0;
    void* reserve = force_pageable ? nullptr : host_alloc_pinned((size_t)1 << 30);
    c->kv_host.assign((size_t)L, nullptr);
    c->kv_pinned.assign((size_t)L, false);
    int64_t pinned_kv = 0;
    for (int64_t j = 0; j < L; ++j) {
      void* h = nullptr;
      if (!force_pageable && reserve &&
          (pol.pinned_budget_bytes == 0 || pinned_kv + per_layer <= pol.pinned_budget_bytes))
        h = host_alloc_pinned((size_t)per_layer);
      if (h) {
        c->pinned.push_back(h);
        c->pinned_bytes += per_layer;
        pinned_kv += per_layer;
        c->kv_pinned[j] = true;
      } else {
        h = std::aligned_alloc(4096, (size_t)per_layer);
        if (!h) {
          host_free_pinned(reserve);
          set_error("host allocation of %lld bytes for the KV cache failed", (long long)per_layer);
          return PIPO_ERR_OOM_HOST;
        }
        c->kv_pageable.push_back((char*)h);
        c->pool->fill(h, 0, (size_t)per_layer);  // fault the pages in now
      }
      c->kv_host[j] = (char*)h;
    }
    host_free_pinned(reserve);
  }
  c->stats.hbm_bytes = c->hbm_bytes;
  c->stats.pinned_host_bytes = c->pinned_bytes;
  return PIPO_OK;
}

static pipo_status stage_tokens(pipo_ctx* c, const int32_t* tokens, int64_t n) {
  for (int64_t i = 0; i < n; ++i) {
    if (tokens[i] < 0 || tokens[i] >= c->sh.vocab) {
      set_error("token id %d at %lld outside [0, %d)", tokens[i], (long long)i, c->sh.vocab);
      return PIPO_ERR_ARG;
    }
  }
  if (c->pol.embed_on_host) {
    // a prompt's rows (470 MB for a batch of 64 x 512 at d = 7168) on
    // several threads, a decode step's few rows on this one
    par_gather(c->emb_stage, c->tok_host, tokens, n, (size_t)c->d * 2);
  } else {
    std::memcpy(c->ids_stage, tokens, (size_t)n * 4);
  }
  return PIPO_OK;
}

// union of [a, b) intervals clipped to [lo, hi)
static double interval_union(std::vector<std::pair<double, double>>& iv, double lo, double hi) {
  std::sort(iv.begin(), iv.end());
  double total = 0, cur_a = 0, cur_b = -1e300;
  bool open = false;
  for (auto& [a0, b0] : iv) {
    const double a = std::max(a0, lo), b = std::min(b0, hi);
    if (b <= a) continue;
    if (!open || a > cur_b) {
      if (open) total += cur_b - cur_a;
      cur_a = a;
      cur_b = b;
      open = true;
    } else {
      cur_b = std::max(cur_b, b);
    }
  }
  if (open) total += cur_b - cur_a;
  return total;
}

static pipo_status resolve_timeline(pipo_ctx* c) {
  if (!c->timestamps || c->trec.empty()) return PIPO_OK;
  for (int i = 0; i < kNumStreams; ++i) PIPO_HIP_TRY(hipStreamSynchronize(c->st[i]));
  hipEvent_t ref = c->trec.front().a;
  const auto t = [&](hipEvent_t e, double* ms) -> pipo_status {
    float v = 0;
    PIPO_HIP_TRY(hipEventElapsedTime(&v, ref, e));
    *ms = v;
    return PIPO_OK;
  };
  double lo = 1e300, hi = -1e300;
  std::vector<std::pair<double, double>> copies, kernels, all;
  for (const TimedRec& r : c->trec) {
    double a, b;
    PIPO_TRY(t(r.a, &a));
    PIPO_TRY(t(r.b, &b));
    if (r.kind == 3) {
      lo = std::min(lo, a);
      hi = std::max(hi, b);
    } else if (r.kind == 0) {
      kernels.push_back({a, b});
      all.push_back({a, b});
      c->kstat_n[r.cls]++;
      c->kstat_ms[r.cls] += b - a;
      c->kstat_bytes[r.cls] += r.bytes;
      c->kstat_flops[r.cls] += r.flops;
    } else {
      if (r.kind == 1) copies.push_back({a, b});
      all.push_back({a, b});
    }
  }
  if (hi > lo) {
    c->stats.window_ms += hi - lo;
    c->stats.copy_busy_ms += interval_union(copies, lo, hi);
    c->stats.kernel_busy_ms += interval_union(kernels, lo, hi);
    c->stats.busy_ms += interval_union(all, lo, hi);
  }
  c->trec.clear();
  c->tpool_used = 0;
  return PIPO_OK;
}

}  // namespace pipo

// ---------------------------------------------------------------------------
// C ABI
extern "C" {

const char* pipo_last_error(void) { return pipo::g_err.c_str(); }

void* pipo_host_alloc(size_t bytes) { return pipo::host_alloc_pinned(bytes); }
void pipo_host_free(void* p) { pipo::host_free_pinned(p); }

pipo_status pipo_create(const pipo_shape* shape, const pipo_host_weights* weights,
                        const pipo_policy* policy, pipo_ctx** out) {
  clear_error();
  if (!out) {
    set_error("out is NULL");
    return PIPO_ERR_ARG;
  }
  *out = nullptr;
  pipo_ctx* c = nullptr;
  const pipo_status s = guarded([&] {
    c = new pipo_ctx();
    return create_ctx(shape, weights, policy, c);
  });
  if (s != PIPO_OK) {
    destroy_ctx(c);
    return s;
  }
  *out = c;
  return PIPO_OK;
}

void pipo_destroy(pipo_ctx* c) { destroy_ctx(c); }

pipo_status pipo_prefill(pipo_ctx* c, const int32_t* tokens, int32_t b, int32_t P,
                         float* logits_out, int32_t* next_out) {
  clear_error();
  if (!c || !tokens || !next_out) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  if (b < 1 || b > c->pol.max_batch || P < 1 || P > c->pol.max_seq) {
    set_error("prefill b=%d P=%d outside max_batch=%d max_seq=%d", b, P, c->pol.max_batch,
              c->pol.max_seq);
    return PIPO_ERR_ARG;
  }
  if (c->failed) {
    set_error("an earlier pass failed part way; the context must be destroyed");
    return PIPO_ERR_STATE;
  }
  return guarded([&]() -> pipo_status {
    PIPO_HIP_TRY(hipSetDevice(c->device));
    const auto t0 = std::chrono::steady_clock::now();
    c->have_seq = false;
    c->b = b;
    // tokens[b][P] -> row i * P + p, the order the kernels use
    PIPO_TRY(stage_tokens(c, tokens, (int64_t)b * P));
    c->pass = PassInfo{true, 0, P, (int64_t)b * c->kv_row};
    PIPO_TRY(run_pass(c, logits_out, next_out, false));
    c->pos = P;
    c->have_seq = true;
    c->stats.prefill_wall_ms =
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    return PIPO_OK;
  });
}

pipo_status pipo_decode_step(pipo_ctx* c, const int32_t* tokens, float* logits_out,
                             int32_t* next_out) {
  clear_error();
  if (!c || !tokens || !next_out) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  if (c->failed) {
    set_error("an earlier pass failed part way; the context must be destroyed");
    return PIPO_ERR_STATE;
  }
  if (!c->have_seq) {
    set_error("decode before prefill");
    return PIPO_ERR_STATE;
  }
  if (c->pos >= c->pol.max_seq) {
    set_error("sequences already hold max_seq=%d positions", c->pol.max_seq);
    return PIPO_ERR_STATE;
  }
  return guarded([&]() -> pipo_status {
    PIPO_HIP_TRY(hipSetDevice(c->device));
    const auto t0 = std::chrono::steady_clock::now();
    PIPO_TRY(stage_tokens(c, tokens, c->b));
    c->pass = PassInfo{false, c->pos, 1, (int64_t)c->b * c->kv_row};
    PIPO_TRY(run_pass(c, logits_out, next_out, true));
    c->pos += 1;
    c->stats.decode_steps++;
    c->stats.decode_wall_ms +=
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    return PIPO_OK;
  });
}

pipo_status pipo_get_stats(pipo_ctx* c, pipo_stats* out) {
  clear_error();
  if (!c || !out) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  return guarded([&]() -> pipo_status {
    PIPO_HIP_TRY(hipSetDevice(c->device));
    PIPO_TRY(resolve_timeline(c));
    *out = c->stats;
    int n = 0;
    for (int k = 0; k < kNumKernels * 2 && n < PIPO_MAX_KERNEL_STATS; ++k) {
      if (c->kstat_n[k] == 0) continue;
      pipo_kernel_stat& ks = out->kernels[n++];
      std::snprintf(ks.name, sizeof ks.name, "%s_%s", kKernelNames[k / 2],
                    (k & 1) ? "prefill" : "decode");
      ks.launches = c->kstat_n[k];
      ks.total_ms = c->kstat_ms[k];
      ks.alg_bytes = c->kstat_bytes[k];
      ks.alg_flops = c->kstat_flops[k];
    }
    out->n_kernel_stats = n;
    return PIPO_OK;
  });
}

pipo_status pipo_debug_fail_pass(pipo_ctx* c, int64_t n_ops) {
  clear_error();
  if (!c) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  c->fail_after_ops = n_ops < 0 ? -1 : n_ops;
  return PIPO_OK;
}

pipo_status pipo_set_timestamps(pipo_ctx* c, int32_t on) {
  clear_error();
  if (!c) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  return guarded([&]() -> pipo_status {
    PIPO_HIP_TRY(hipSetDevice(c->device));
    PIPO_TRY(resolve_timeline(c));
    c->timestamps = on != 0;
    return PIPO_OK;
  });
}

pipo_status pipo_reset_stats(pipo_ctx* c) {
  clear_error();
  if (!c) {
    set_error("NULL argument");
    return PIPO_ERR_ARG;
  }
  PIPO_HIP_TRY(hipSetDevice(c->device));
  for (int i = 0; i < kNumStreams; ++i) PIPO_HIP_TRY(hipStreamSynchronize(c->st[i]));
  c->trec.clear();
  c->tpool_used = 0;
  const int64_t hbm = c->stats.hbm_bytes, pin = c->stats.pinned_host_bytes;
  c->stats = pipo_stats{};
  c->stats.hbm_bytes = hbm;
  c->stats.pinned_host_bytes = pin;
  for (int k = 0; k < kNumKernels * 2; ++k) {
    c->kstat_n[k] = 0;
    c->kstat_ms[k] = c->kstat_bytes[k] = c->kstat_flops[k] = 0;
  }
  return PIPO_OK;
}

// `bytes` pinned -> HBM per round as consecutive copies of `chunk` bytes,
// copy k on stream k % n_streams (the pipeline's pattern); best round
static pipo_status measure_h2d(int64_t bytes, int64_t chunk, int32_t iters, int32_t n_streams,
                               double* gbps) {
  if (bytes <= 0 || chunk <= 0 || iters < 1 || n_streams < 1 || n_streams > 2 || !gbps) {
    set_error("invalid arguments");
    return PIPO_ERR_ARG;
  }
  void* h = pipo::host_alloc_pinned((size_t)bytes);
  if (!h) {
    set_error("pinned allocation of %lld bytes failed", (long long)bytes);
    return PIPO_ERR_OOM_HOST;
  }
  std::memset(h, 1, (size_t)bytes);
  void* dptr = nullptr;
  if (hipMalloc(&dptr, (size_t)bytes) != hipSuccess) {
    (void)hipGetLastError();
    pipo::host_free_pinned(h);
    set_error("hipMalloc of %lld bytes failed", (long long)bytes);
    return PIPO_ERR_OOM_DEVICE;
  }
  hipStream_t st[2] = {};
  hipEvent_t e0 = nullptr, e1 = nullptr, ej = nullptr;
  pipo_status status = PIPO_OK;
  double best = 0;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess ||
      hipEventCreateWithFlags(&ej, hipEventDisableTiming) != hipSuccess) {
    set_error("hipEventCreate failed");
    status = PIPO_ERR_HIP;
  }
  for (int i = 0; i < n_streams && status == PIPO_OK; ++i)
    if (hipStreamCreateWithFlags(&st[i], hipStreamNonBlocking) != hipSuccess) status = PIPO_ERR_HIP;
  for (int it = 0; it <= iters && status == PIPO_OK; ++it) {  // first round warms up
    bool ok = hipEventRecord(e0, st[0]) == hipSuccess;
    if (n_streams == 2) ok = ok && hipStreamWaitEvent(st[1], e0, 0) == hipSuccess;
    int k = 0;
    for (int64_t a = 0; a < bytes && ok; a += chunk, ++k) {
      const int64_t n = std::min(chunk, bytes - a);
      ok = hipMemcpyAsync((char*)dptr + a, (char*)h + a, (size_t)n, hipMemcpyHostToDevice,
                          st[k % n_streams]) == hipSuccess;
    }
    if (n_streams == 2) {
      ok = ok && hipEventRecord(ej, st[1]) == hipSuccess &&
           hipStreamWaitEvent(st[0], ej, 0) == hipSuccess;
    }
    ok = ok && hipEventRecord(e1, st[0]) == hipSuccess && hipEventSynchronize(e1) == hipSuccess;
    float ms = 0;
    ok = ok && hipEventElapsedTime(&ms, e0, e1) == hipSuccess;
    if (!ok) {
      set_error("h2d probe: HIP call failed");
      status = PIPO_ERR_HIP;
      break;
    }
    if (it > 0 && ms > 0) best = std::max(best, (double)bytes / (ms * 1e-3) / 1e9);
  }
  for (int i = 0; i < 2; ++i)
    if (st[i]) (void)hipStreamDestroy(st[i]);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (ej) (void)hipEventDestroy(ej);
  (void)hipFree(dptr);
  pipo::host_free_pinned(h);
  *gbps = best;
  return status;
}

pipo_status pipo_measure_h2d_peak(int64_t bytes, int32_t iters, int32_t n_streams, double* gbps) {
  clear_error();
  if (n_streams < 1) {
    set_error("invalid arguments");
    return PIPO_ERR_ARG;
  }
  return measure_h2d(bytes, pipo::align_up((bytes + n_streams - 1) / n_streams, 4096), iters,
                     n_streams, gbps);
}

pipo_status pipo_measure_h2d_chunked(int64_t bytes, int64_t chunk_bytes, int32_t iters,
                                     int32_t n_streams, double* gbps) {
  clear_error();
  return measure_h2d(bytes, chunk_bytes, iters, n_streams, gbps);
}

pipo_status pipo_measure_disk_tier(pipo_ctx* c, int64_t bytes, int32_t iters, double* gbps) {
  clear_error();
  if (!c || !gbps || bytes <= 0 || iters < 1) {
    set_error("measure_disk_tier: bad arguments");
    return PIPO_ERR_ARG;
  }
  if (c->disk_fd < 0) {
    set_error("measure_disk_tier: the context has no disk tier");
    return PIPO_ERR_STATE;
  }
  return guarded([&]() -> pipo_status {
    PIPO_HIP_TRY(hipSetDevice(c->device));
    for (int i = 0; i < kNumStreams; ++i) PIPO_HIP_TRY(hipStreamSynchronize(c->st[i]));
    StagingRing& r = c->stage_h2d;
    const int64_t total = std::min(align_up(bytes, 4096), c->L * c->layer_bytes);
    double best = 0;
    for (int it = 0; it < iters; ++it) {
      const auto t0 = std::chrono::steady_clock::now();
      for (int64_t off = 0; off < total; off += r.buf_bytes) {
        const int64_t n = std::min(r.buf_bytes, total - off);
        if (!c->pool->pread_all(c->disk_fd, r.buf[0], (size_t)n, off,
                                c->disk_direct ? c->disk_bounce : nullptr)) {
          set_error("measure_disk_tier: reading failed: %s", std::strerror(errno));
          return PIPO_ERR_IO;
        }
      }
      const double sec =
          std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
      best = std::max(best, (double)total / sec / 1e9);
    }
    *gbps = best;
    return PIPO_OK;
  });
}

pipo_status pipo_measure_disk_read(const char* dir, int64_t bytes, int64_t chunk_bytes,
                                   int32_t n_threads, int32_t iters, double* gbps,
                                   int32_t* direct) {
  clear_error();
  if (!gbps || bytes <= 0 || chunk_bytes <= 0 || n_threads < 1 || n_threads > 64 || iters < 1) {
    set_error("measure_disk_read: bad arguments");
    return PIPO_ERR_ARG;
  }
  chunk_bytes = align_up(chunk_bytes, 4096);
  bytes = align_up(bytes, chunk_bytes);
  std::unique_ptr<CopyPool> pool;
  PIPO_TRY(guarded([&] {
    pool.reset(new CopyPool(n_threads));
    return PIPO_OK;
  }));
  const std::string d = dir && dir[0] ? dir : ".";
  std::string path = d + "/pipo_probe_XXXXXX";
  int fd = ::mkstemp(&path[0]);
  if (fd < 0) {
    set_error("measure_disk_read: cannot create a file in %s: %s", d.c_str(), std::strerror(errno));
    return PIPO_ERR_IO;
  }
  const int fdd = ::open(path.c_str(), O_RDWR | O_DIRECT);
  bool is_direct = false;
  if (fdd >= 0) {
    ::close(fd);
    fd = fdd;
    is_direct = true;
  }
  ::unlink(path.c_str());
  char* buf = static_cast<char*>(std::aligned_alloc(4096, (size_t)chunk_bytes));
  char* bounce = static_cast<char*>(std::aligned_alloc(4096, (size_t)chunk_bytes));
  pipo_status st = PIPO_OK;
  if (!buf || !bounce) {
    set_error("measure_disk_read: host allocation failed");
    st = PIPO_ERR_OOM_HOST;
  }
  if (st == PIPO_OK) {
    std::memset(buf, 0x5a, (size_t)chunk_bytes);
    for (int64_t off = 0; off < bytes && st == PIPO_OK; off += chunk_bytes)
      if (!pool->pwrite_all(fd, buf, (size_t)chunk_bytes, off)) {
        set_error("measure_disk_read: writing %s failed: %s", d.c_str(), std::strerror(errno));
        st = PIPO_ERR_IO;
      }
  }
  double best = 0;
  for (int it = 0; it < iters && st == PIPO_OK; ++it) {
    const auto t0 = std::chrono::steady_clock::now();
    for (int64_t off = 0; off < bytes && st == PIPO_OK; off += chunk_bytes)
      if (!pool->pread_all(fd, buf, (size_t)chunk_bytes, off, is_direct ? bounce : nullptr)) {
        set_error("measure_disk_read: reading %s failed: %s", d.c_str(), std::strerror(errno));
        st = PIPO_ERR_IO;
      }
    const double sec =
        std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    best = std::max(best, (double)bytes / sec / 1e9);
  }
  ::close(fd);
  std::free(buf);
  std::free(bounce);
  if (st != PIPO_OK) return st;
  *gbps = best;
  if (direct) *direct = is_direct ? 1 : 0;
  return PIPO_OK;
}

}  // extern "C"
