/*
 * pipo.h -- C ABI of an MI355X (gfx950) pipelined-offloading decoder.
 *
 * The library runs the forward pass of an OPT-style decoder (pre-LN blocks:
 * LayerNorm, QKV projection, causal softmax attention over a KV cache,
 * output projection, LayerNorm, ReLU MLP; tied output head; greedy
 * decoding) on one GPU while the weights of each layer -- and, optionally,
 * its KV cache -- live in pinned host memory and are streamed into HBM a
 * few layers ahead of the computation.  This is the pipelined offloading of
 * PIPO (Liu, Li, Li; arXiv 2504.03664):
 *   - weights are loaded layer by layer and released after use
 *     (Section 3.1.1), in fine-grained chunks of merged per-layer tensors
 *     (Section 3.3, blockwise transfer and data merging);
 *   - four task types -- computation, weight loading, KV-cache loading and
 *     KV-cache saving -- overlap, each load finishing before its layer
 *     computes and each save finishing before the same layer loads its
 *     cache at the next token (Section 3.1.2; Section 3.2.2, Algorithm 1);
 *   - loading runs ahead of computation so that two or more layers are
 *     resident (Section 3.2.3, performance-optimized pipeline);
 *   - INT4 weights are consumed directly by the GEMM (Section 3.4).
 * A second model family, LLaMA 3.1 (the paper's other evaluated models,
 * Section 4.1; memory model of Section 3.5), runs through the same
 * pipeline: RMSNorm, grouped-query attention with rotary positions,
 * a SwiGLU MLP, untied output head, no biases (see pipo_shape).
 * The lifecycle follows the paper's workflow (Algorithm 2): pipo_create
 * initialises the model data, the transfer machinery and the schedule;
 * pipo_prefill and pipo_decode_step run the generation loop.
 *
 * Conventions for every entry point:
 *   - fp16 values are passed as their IEEE binary16 bit patterns (uint16_t);
 *   - matrices are row-major [out][in] ("N rows of K inputs");
 *   - host pointers are plain CPU pointers; "device" pointers are HBM
 *     addresses on the current HIP device;
 *   - every call returns a pipo_status (no exceptions cross the ABI); on
 *     failure pipo_last_error() describes it;
 *   - a context is used by one host thread at a time.
 */
#ifndef PIPO_H
#define PIPO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PIPO_OK = 0,
  PIPO_ERR_ARG = -1,          /* invalid argument or shape */
  PIPO_ERR_OOM_DEVICE = -2,   /* HBM allocation failed or exceeds hbm_budget_bytes */
  PIPO_ERR_OOM_HOST = -3,     /* host allocation failed (pinned memory or heap) */
  PIPO_ERR_HIP = -4,          /* a HIP runtime call failed */
  PIPO_ERR_STATE = -5,        /* call not valid in the context's state */
  PIPO_ERR_UNSUPPORTED = -6,  /* shape or policy outside what the kernels support */
  PIPO_ERR_IO = -7            /* a file operation of the disk tier failed */
} pipo_status;
/* No entry point lets a C++ exception escape: an exhausted host heap inside
 * any call that returns pipo_status is reported as PIPO_ERR_OOM_HOST, in
 * addition to the errors each call lists; a helper thread that the system
 * refuses makes the call do that share of its host work on the calling
 * thread instead. */

/* Weight storage format of the four per-layer matrices. */
enum { PIPO_W_FP16 = 0, PIPO_W_INT4_G64 = 1 };

/* KV cache storage format.  PIPO_KV_INT4_G64 (Section 2: the KV cache may
 * be kept in 4 bits like the weights): a cached key or value row of d
 * elements takes d/2 code bytes (element 2i in the low nibble of byte i)
 * followed by d/64 fp16 (scale, min) pairs, one per 64 consecutive
 * elements, 9d/16 bytes in all instead of 2d.  A new row (fp16) is
 * quantized when it is written: per group, in fp32, scale = fp16((max -
 * min) / 15), min = fp16(min), code = clamp(rint((x - min) / scale), 0, 15)
 * rounding half to even (0 where scale is 0); every attention, prefill
 * included, reads code * scale + min.  Needs d_model % 256 == 0. */
enum { PIPO_KV_FP16 = 0, PIPO_KV_INT4_G64 = 1 };

/* pipo_policy.debug_flags */
enum {
  PIPO_DBG_POISON_SLOTS = 1,  /* fill a weight/KV slot with NaN before every refill */
  PIPO_DBG_COPY_DELAY = 2,    /* host-side sleep of copy_delay_us before every chunk copy */
  PIPO_DBG_TIMESTAMPS = 4,    /* record device timestamps of copies and kernels (stats) */
  PIPO_DBG_KV_PAGEABLE = 8,   /* keep the host KV cache in pageable memory (staged copies) */
  PIPO_DBG_SEGMENT_COPIES = 16, /* copy each tensor of a layer on its own, even where the
                                   layer's matrices could be copied as one merged range */
  PIPO_DBG_UNFUSED = 32         /* run the LLaMA SwiGLU as its own kernel after the gate/up
                                   GEMM also at decode, where it is otherwise that GEMM's
                                   epilogue (same values; for tests) */
};

/* Model families (pipo_shape.family).
 *  PIPO_FAMILY_OPT: pre-LN blocks with LayerNorm (gain and bias), learned
 *    positions added to the token embedding, multi-head attention, biases on
 *    every projection, ReLU MLP (w1 [d_ffn][d], w2 [d][d_ffn]), final
 *    LayerNorm, output head tied to the token table.
 *  PIPO_FAMILY_LLAMA: pre-norm blocks with RMSNorm (y = x / sqrt(mean(x^2) +
 *    eps) * g); q, k, v without biases; rotary positions on q and k, pairing
 *    element i with i + head_dim/2 of every head at angle p * w_i, w_i =
 *    rope_theta^(-2i/head_dim), with the LLaMA 3.1 frequency scaling when
 *    rope_factor > 0 (a component whose wavelength 2 pi / w_i exceeds
 *    rope_orig_max_pos / rope_low_freq_factor is divided by rope_factor, one
 *    shorter than rope_orig_max_pos / rope_high_freq_factor is kept, in
 *    between w' = (1 - s) w / rope_factor + s w with s = (rope_orig_max_pos
 *    / wavelength - low) / (high - low)); keys are cached after rotation;
 *    grouped-query attention (query head h reads key/value head h / (n_heads
 *    / n_kv_heads)); SwiGLU MLP h = silu(x w_gate^T) * (x w_up^T) with gate
 *    and up stacked in w1 [2 d_ffn][d] (gate rows first), then h w2^T;
 *    final RMSNorm; untied output head (pipo_host_weights.lm_head).
 * Both: q is scaled by head_dim^-1/2, causal softmax attention, greedy
 * decoding. */
enum { PIPO_FAMILY_OPT = 0, PIPO_FAMILY_LLAMA = 1 };

/* Decoder shape.  Constraints: d_model = n_heads * head_dim with head_dim
 * 64 or 128; d_model and d_ffn multiples of 128; vocab >= 1; n_heads a
 * multiple of n_kv_heads, 1, 2, 4 or 8 query heads per key/value head.
 * The fields after ln_eps are zero for OPT. */
typedef struct {
  int32_t n_layers, d_model, n_heads, d_ffn, vocab;
  int32_t max_pos;      /* OPT: positions the learned table covers (rows = max_pos +
                           pos_offset); LLaMA: longest sequence the rotary table covers */
  int32_t pos_offset;   /* OPT: row of position 0 in the position table (2); LLaMA: unused */
  float ln_eps;         /* LayerNorm / RMSNorm epsilon (1e-5) */
  int32_t family;       /* PIPO_FAMILY_OPT (0) or PIPO_FAMILY_LLAMA */
  int32_t n_kv_heads;   /* key/value heads; 0 means n_heads (OPT: must be 0 or n_heads) */
  float rope_theta;     /* LLaMA: rotary base (500000 for LLaMA 3.1) */
  float rope_factor;    /* LLaMA: 3.1 frequency scaling factor (8), 0 for none */
  float rope_low_freq_factor, rope_high_freq_factor;  /* LLaMA 3.1: 1 and 4 */
  int32_t rope_orig_max_pos;  /* LLaMA 3.1: 8192 (used when rope_factor > 0) */
} pipo_shape;

/* One group-wise INT4 matrix W[N][K]: W[n][k] = code * scale + min, one
 * (scale, min) pair per 64 consecutive k of a row (Section 3.4 keeps the
 * weights in 4 bits; the grouping is the workload's definition). */
typedef struct {
  const uint8_t* q;           /* [N][K/2]; code(2i) in the low nibble of byte i */
  const uint16_t* scale_min;  /* [N][K/64][2] fp16: {scale, min} */
} pipo_q4;

/* Host tensors of one layer (caller-owned; read, never written).  With
 * dkv = n_kv_heads * head_dim (= d without grouped-query attention) and
 * F = d_ffn.  LLaMA uses only ln1_g, ln2_g and the matrices (the bias and
 * LayerNorm-bias pointers are ignored). */
typedef struct {
  const uint16_t *ln1_g, *ln1_b;   /* [d] */
  const uint16_t *bqkv;            /* [3d]: q, k, v biases */
  const uint16_t *bo;              /* [d] */
  const uint16_t *ln2_g, *ln2_b;   /* [d] */
  const uint16_t *b1;              /* [d_ffn] */
  const uint16_t *b2;              /* [d] */
  const uint16_t *wqkv;            /* [d + 2 dkv][d] rows: q, k, v          (PIPO_W_FP16) */
  const uint16_t *wo;              /* [d][d]                                (PIPO_W_FP16) */
  const uint16_t *w1;              /* OPT [F][d]; LLaMA [2F][d] gate, up    (PIPO_W_FP16) */
  const uint16_t *w2;              /* [d][F]                                (PIPO_W_FP16) */
  pipo_q4 qqkv, qo, q1, q2;        /* same matrices                         (PIPO_W_INT4_G64) */
} pipo_layer_host;

/* Layout of the four layer matrices in pipo_host_weights (pipo_host_weights.layout).
 *  PIPO_LAYOUT_ROW_MAJOR: W[N][K] row-major; INT4 as pipo_q4 describes.
 *  PIPO_LAYOUT_FRAGMENT: the layout the decode kernels read fastest (one
 *    contiguous 1 KiB per wave load; pipo_pack_f16 / pipo_pack_w4 produce
 *    it): fp16 W in blocks of 16 rows x 32 k, block (rg, kb) at halves
 *    512 (rg K/32 + kb), inside which the 16 bytes at 16 (r + 16 g) hold
 *    W[16 rg + r][32 kb + 8 g .. + 7]; INT4 codes in blocks of 16 rows x
 *    128 k, block (rg, kb) at byte 1024 (rg K/128 + kb), the 16 bytes at
 *    16 (r + 16 g) holding row 16 rg + r's codes for k = 128 kb + 32 g ..
 *    + 31 (nibble order as row-major); (scale, min) pairs in 32-pair
 *    blocks, pair 32 (rg K/128 + kb) + 2 r + j = row 16 rg + r, group
 *    2 kb + j.  Every layer matrix has N % 16 == 0 and K % 128 == 0.
 * With row-major input the library converts what it copies (its own
 * pinned regions, resident HBM copies, the disk tier's file); matrices it
 * would stream in place from pipo_host_alloc memory keep the row-major
 * layout for the whole context.  The output head is always row-major. */
enum { PIPO_LAYOUT_ROW_MAJOR = 0, PIPO_LAYOUT_FRAGMENT = 1 };

typedef struct {
  const uint16_t* tok_emb;   /* [vocab][d]; OPT: also the output head (tied) */
  const uint16_t* pos_emb;   /* OPT: [max_pos + pos_offset][d]; LLaMA: unused */
  const uint16_t *lnf_g, *lnf_b;   /* final norm [d] (LLaMA: lnf_b unused) */
  const pipo_layer_host* layers;   /* [n_layers] */
  const uint16_t* lm_head;   /* LLaMA: output head [vocab][d]; OPT: unused */
  int32_t layout;            /* PIPO_LAYOUT_* of the layer matrices */
} pipo_host_weights;

/* Offload policy (the paper's (S_off, S_pipe) pair, Algorithm 2, made
 * explicit).  Zero-initialise and set what you need; 0 picks the default. */
typedef struct {
  int32_t wfmt;              /* PIPO_W_FP16 or PIPO_W_INT4_G64 */
  int32_t weights_on_host;   /* 1: stream every layer each pass; 0: all layers resident in HBM */
  int32_t embed_on_host;     /* 1: stream the output head each pass, gather embeddings on the
                                host; 0: token table (and an untied head) resident in HBM */
  int32_t kv_on_host;        /* 1: KV cache in library-owned host memory (pinned where
                                possible, see pinned_budget_bytes), each layer's prefix loaded
                                before its attention and the new rows saved after it (a call
                                returns with its rows saved); 0: KV cache resident in HBM */
  int32_t n_weight_slots;    /* HBM slots the layers rotate through (default 3, 1..16).  3: the
                                performance-optimized pipeline (Section 3.2.3) -- loads run two
                                units ahead; 1: the memory-efficient pipeline -- one layer's
                                weights (and KV buffer) in HBM, a unit's load waits until the
                                previous unit's compute (and KV save) is done */
  int32_t n_h2d_streams;     /* host-to-device copy streams (default 2, max 2); chunk k goes
                                to stream k % n, so one DMA is always queued behind another */
  int64_t chunk_bytes;       /* bytes per copy chunk (default 64 MiB; rounded to 4 KiB) */
  int32_t max_batch;         /* sequences per pass (>= 1) */
  int32_t max_seq;           /* prompt + generated positions per sequence (<= max_pos) */
  int64_t hbm_budget_bytes;  /* 0: unlimited; else pipo_create fails with OOM_DEVICE above it */
  int32_t debug_flags;       /* PIPO_DBG_* */
  int32_t copy_delay_us;     /* delay for PIPO_DBG_COPY_DELAY */
  int64_t pinned_budget_bytes; /* 0: pin host KV layers while the system grants pinned memory;
                                  else at most this many bytes of pinned host KV.  KV layers
                                  that are not pinned live in pageable memory and move through
                                  pinned staging buffers, copied by host worker threads (the
                                  paper's multi-thread transfer, Section 3.3) */
  int32_t copy_threads;      /* host threads for staged copies and disk reads (default 8) */
  int32_t kv_fmt;            /* PIPO_KV_FP16 (default) or PIPO_KV_INT4_G64 */
  int32_t weights_on_disk;   /* 1: the disk tier (Section 3.1.1 offloads to CPU memory or disk;
                                Section 3.3's blockwise transfer): pipo_create writes every
                                layer unit to a library-owned file in disk_dir (removed when the
                                context is destroyed; the caller's layer tensors are read only
                                during pipo_create) and each pass streams the layers disk ->
                                pinned staging -> HBM in chunk_bytes pieces, read by
                                copy_threads threads with direct I/O where the file system
                                allows it, the next chunk's read overlapping the previous
                                chunk's DMA.  Requires weights_on_host.  The output head stays
                                in host memory (embed_on_host) or HBM. */
  int32_t reserved0;         /* 0 */
  const char* disk_dir;      /* directory of the disk tier's file (NULL: the working directory) */
} pipo_policy;

/* The paper's two pipeline options (Section 3.2.3). */
enum { PIPO_PIPE_PERFORMANCE = 0, PIPO_PIPE_MEMORY_EFFICIENT = 1 };

/* What a policy costs (pipo_plan_policy, pipo_configure).  hbm_bytes is the
 * exact sum of the device allocations pipo_create makes for the policy
 * (activations are sized for max_batch x max_seq rows: the prefill peak). */
typedef struct {
  int64_t weight_bytes;        /* W: layer tensors, token and position tables (or token table
                                  and untied head), final norm */
  int64_t kv_bytes;            /* C: KV cache of max_batch x max_seq positions, all layers */
  int64_t hbm_bytes;           /* device memory pipo_create allocates */
  int64_t host_kv_bytes;       /* host memory the library allocates for the KV cache */
  int64_t h2d_bytes_per_step;  /* host-to-device bytes of a decode step at the last position */
  int32_t pipeline;            /* PIPO_PIPE_* (memory-efficient: n_weight_slots == 1) */
  int32_t reserved0;
  int64_t host_weight_bytes;   /* weights that live in host memory (streamed layers unless on
                                  disk, streamed head) plus the disk tier's staging buffers */
  int64_t disk_bytes;          /* the disk tier's file (0 without it) */
  int64_t disk_bytes_per_step; /* bytes a decode step reads from disk */
} pipo_plan;

/* Resources for the automatic configuration. */
typedef struct {
  int64_t hbm_bytes;   /* device memory the context may use; 0: the device's free memory */
  int64_t host_bytes;  /* host memory for the weights kept there and a host KV cache; 0: the
                          system's available memory */
  int64_t disk_bytes;  /* disk space for the disk tier; 0: no disk tier */
} pipo_resources;

/* Per-kernel timing (filled when PIPO_DBG_TIMESTAMPS is set): each launch
 * is bracketed by events on the stream that runs it. */
typedef struct {
  char name[32];
  int64_t launches;
  double total_ms;           /* summed launch durations */
  double alg_bytes;          /* algorithmic bytes summed over launches */
  double alg_flops;          /* algorithmic flops summed over launches */
} pipo_kernel_stat;

#define PIPO_MAX_KERNEL_STATS 16

typedef struct {
  int64_t h2d_bytes;         /* host-to-device bytes issued since the last reset */
  int64_t h2d_weight_bytes;  /*   of which weights (incl. output head) */
  int64_t h2d_kv_bytes;      /*   of which KV-cache prefixes */
  int64_t d2h_bytes;         /* device-to-host bytes (KV saves, tokens, logits) */
  int64_t n_copies;          /* copy commands issued */
  int64_t n_kernels;         /* kernel launches issued */
  int64_t decode_steps;      /* pipo_decode_step calls since the last reset */
  double decode_wall_ms;     /* host wall time inside those calls */
  double prefill_wall_ms;    /* host wall time of the last pipo_prefill */
  /* device timeline of the decode steps since the last reset (PIPO_DBG_TIMESTAMPS) */
  double window_ms;          /* first decode-step start to last decode-step end */
  double copy_busy_ms;       /* union of host-to-device copy intervals inside the window */
  double kernel_busy_ms;     /* union of compute-stream kernel intervals inside the window */
  double busy_ms;            /* union of both */
  int64_t staged_bytes;      /* bytes that went through the pinned staging buffers */
  int64_t disk_read_bytes;   /* bytes read from the disk tier's file */
  double disk_read_ms;       /* host wall time spent in those reads */
  int64_t hbm_bytes;         /* HBM the context holds */
  int64_t pinned_host_bytes; /* pinned host memory the context holds */
  int32_t n_kernel_stats;
  pipo_kernel_stat kernels[PIPO_MAX_KERNEL_STATS];
} pipo_stats;

typedef struct pipo_ctx pipo_ctx;

/*
 * Create a context on the current HIP device.
 *   shape, weights, policy: read during the call.  The matrices in `weights`
 *     must stay valid and unchanged until pipo_destroy when weights_on_host
 *     (or embed_on_host) is set: matrices in pinned memory from
 *     pipo_host_alloc are streamed in place; other host memory is first
 *     copied into library-owned pinned memory.
 *   out: receives the context (NULL on failure).
 * Errors: ARG (bad shape/policy/NULL tensor), UNSUPPORTED (shape outside the
 * kernels' range), OOM_DEVICE, OOM_HOST, HIP.
 */
pipo_status pipo_create(const pipo_shape* shape, const pipo_host_weights* weights,
                        const pipo_policy* policy, pipo_ctx** out);

/*
 * Start b new sequences: run the whole prompt tokens[b][P] (row-major host
 * int32, ids in [0, vocab)), fill the KV cache for positions 0..P-1, and
 * return the greedy next token of each sequence in next_out[b] (host).  If
 * logits_out is not NULL it receives the fp32 logits [b][vocab] of the last
 * prompt position.  Returns once next_out is written.
 * Errors: ARG (b < 1 or > max_batch, P < 1 or > max_seq, id out of range),
 * STATE (an earlier pass of this context failed part way), HIP.
 */
pipo_status pipo_prefill(pipo_ctx* ctx, const int32_t* tokens, int32_t b, int32_t P,
                         float* logits_out, int32_t* next_out);

/*
 * Append one token per sequence (tokens[b], host int32; usually the previous
 * next_out, any id for teacher forcing) at the next position and return the
 * greedy next tokens (next_out[b]) and optionally the fp32 logits [b][vocab].
 * b must equal the prefill's b.
 * Errors: STATE (no prefill yet, the sequences already hold max_seq
 * positions, or an earlier pass of this context failed part way), ARG, HIP.
 */
pipo_status pipo_decode_step(pipo_ctx* ctx, const int32_t* tokens, float* logits_out,
                             int32_t* next_out);

/* Copy the context's counters into *out (see pipo_stats). */
pipo_status pipo_get_stats(pipo_ctx* ctx, pipo_stats* out);

/* Cost of a policy for a shape (no allocation, no device needed).
 * Errors: ARG, UNSUPPORTED (as pipo_create would report them). */
pipo_status pipo_plan_policy(const pipo_shape* shape, const pipo_policy* policy,
                             pipo_plan* plan_out);

/*
 * Automatic configuration (Section 3.5, Eq. (1); Algorithm 2's Configure):
 * choose where the weights, the output head and the KV cache live and which
 * pipeline runs, for a shape, weight and KV formats, max_batch and max_seq
 * within the given resources.  Eq. (1) puts the weights in HBM when they
 * fit, else in host memory, else on disk, and takes the performance-
 * optimized pipeline when its peak memory fits, else the memory-efficient
 * one; here every placement (weights and head resident or streamed, the
 * streamed layers in host memory or on disk when res->disk_bytes allows,
 * KV resident or on the host) and pipeline (3, 2 or 1 slots) is costed
 * exactly and the one that streams the fewest bytes per decode step within
 * the budgets wins; on ties host memory before disk, then more slots.
 * *policy_out gets the choice (with hbm_budget_bytes set to the budget,
 * chunk_bytes and copy streams at their defaults, disk_dir NULL) and, if
 * plan_out is not NULL, its cost.  Errors: ARG, UNSUPPORTED, OOM_DEVICE
 * (not even the memory-efficient pipeline fits), OOM_HOST (what must stay
 * in host memory does not fit, even with the layers on disk), HIP
 * (querying free HBM).
 */
pipo_status pipo_configure(const pipo_shape* shape, int32_t wfmt, int32_t kv_fmt,
                           int32_t max_batch, int32_t max_seq, const pipo_resources* res,
                           pipo_policy* policy_out, pipo_plan* plan_out);

/* Turn device timestamps (PIPO_DBG_TIMESTAMPS) on or off between calls.
 * While on, every copy and kernel is bracketed by two events and each pass
 * ends by synchronising all of the context's streams (which stops the next
 * call's loads from running ahead); figures recorded so far are kept. */
pipo_status pipo_set_timestamps(pipo_ctx* ctx, int32_t on);

/* Test hook for failure handling: the context's next pass (prefill or
 * decode step) stops after issuing n_ops of its planned copy and kernel
 * operations and returns PIPO_ERR_HIP, as a failed copy or launch in the
 * middle of a pass would.  Everything already issued still runs to its end
 * (the failing call waits for it).  After any pass that fails part way the
 * context refuses pipo_prefill and pipo_decode_step with PIPO_ERR_STATE
 * until it is destroyed: its schedule had already counted the rest of the
 * pass as issued.  n_ops < 0 clears the hook.  Errors: ARG. */
pipo_status pipo_debug_fail_pass(pipo_ctx* ctx, int64_t n_ops);

/* Zero the counters and timelines of pipo_stats (allocation figures stay). */
pipo_status pipo_reset_stats(pipo_ctx* ctx);

/* Release everything the context holds.  NULL is allowed. */
void pipo_destroy(pipo_ctx* ctx);

/*
 * Host-to-device link probe: copy `bytes` from pinned host memory to HBM
 * `iters` times, split evenly over n_streams (1 or 2) copy streams, and
 * return the best rate in *gbps (1e9 bytes per second).  Allocates and
 * frees its own buffers.  Errors: ARG, OOM_HOST, OOM_DEVICE, HIP.
 */
pipo_status pipo_measure_h2d_peak(int64_t bytes, int32_t iters, int32_t n_streams,
                                  double* gbps);

/*
 * The same probe with the transfer pattern of the pipeline (Section 3.3,
 * blockwise transfer): each round copies `bytes` as consecutive copies of
 * chunk_bytes, copy k on stream k % n_streams, timed from the first copy's
 * start to the last one's end; best of `iters` rounds.  Used to choose
 * pipo_policy.chunk_bytes.  Errors: ARG, OOM_HOST, OOM_DEVICE, HIP.
 */
pipo_status pipo_measure_h2d_chunked(int64_t bytes, int64_t chunk_bytes, int32_t iters,
                                     int32_t n_streams, double* gbps);

/*
 * Disk probe for the disk tier: write a file of `bytes` in `dir` (removed
 * again), then read it `iters` times in chunk_bytes pieces with n_threads
 * threads the way the disk tier does (direct I/O where the file system
 * allows it, through a pageable buffer) and return the best rate in *gbps
 * (1e9 bytes per second) and whether direct I/O was used in *direct (may be
 * NULL).  Host memory only; no GPU needed.  Errors: ARG, IO, OOM_HOST.
 */
pipo_status pipo_measure_disk_read(const char* dir, int64_t bytes, int64_t chunk_bytes,
                                   int32_t n_threads, int32_t iters, double* gbps,
                                   int32_t* direct);

/* Row-major -> PIPO_LAYOUT_FRAGMENT on the host (caller buffers, not
 * overlapping): fp16 W[N][K] into out (N*K halves), or INT4 codes and
 * (scale, min) pairs into q_out (N*K/2 bytes) and scale_min_out (N*K/32
 * halves).  Errors: ARG (NULL, aliasing, N % 16, K % 32 (fp16) or K % 128
 * (INT4) not 0). */
pipo_status pipo_pack_f16(const uint16_t* W, uint16_t* out, int64_t N, int64_t K);
pipo_status pipo_pack_w4(const uint8_t* q, const uint16_t* scale_min, uint8_t* q_out,
                         uint16_t* scale_min_out, int64_t N, int64_t K);

/* The read rate of a context's own disk-tier file: its first `bytes`
 * (whole layer units in slot layout) read `iters` times exactly as the
 * decode passes read them (chunk_bytes pieces, copy_threads threads, direct
 * I/O through the pageable buffer into pinned staging, no DMA); best rate
 * in *gbps.  Waits for the context's streams first.  Errors: ARG, STATE
 * (no disk tier), IO, HIP. */
pipo_status pipo_measure_disk_tier(pipo_ctx* ctx, int64_t bytes, int32_t iters, double* gbps);

/* Pinned (page-locked) host memory, 4 KiB aligned; NULL on failure.
 * Matrices placed here are streamed by the copy engines without staging. */
void* pipo_host_alloc(size_t bytes);
void pipo_host_free(void* p);

/* Text of the last error on the calling thread ("" if none). */
const char* pipo_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PIPO_H */
