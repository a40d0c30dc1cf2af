/*
 * tpstage.h -- C ABI of one pipeline stage of GPT pre-LN decoder layers on
 * one MI355X (gfx950), with per-tensor keep / recompute / offload policies.
 *
 * Method (paper: "Enhancing Memory Efficiency in LLM Training Through
 * Chronos-aware Pipeline Parallelism", arXiv 2503.03182):
 *   - a pipeline stage runs forward tasks F(mb) and backward tasks B(mb) per
 *     micro-batch; one activation tensor enters/leaves per task (Section 2.1);
 *   - recomputation keeps checkpoints and regenerates the other activations
 *     before they are needed in the backward pass (Section 2.2); T-Recomp
 *     replays the whole recomputed block as a separate step that runs before
 *     the dependent backward (Section 4.2, "Addressing the Concerns"),
 *     while the conventional layer-grouped form replays one group just in
 *     time (Section 4.2, "Concerns Regarding T-Recomp");
 *   - offloading parks tensors in host DRAM and brings them back (Section
 *     2.2); T-Offload moves model state between host and device around the
 *     compute (Section 5); CPU activation offloading composes with it
 *     (Section 5, "Compatibility of T-Offload").
 *
 * Conventions
 *   T = micro_batch * seq tokens; activations are token-major row-major
 *   [T, width] (row r = batch_index * seq + position); weights are [out, in]
 *   row-major (y = x W^T + b); the packed qkv tensor is [T, 3h] with q, k, v
 *   in column blocks [0,h), [h,2h), [2h,3h) and head n at columns n*d..n*d+d-1
 *   of each block.  Storage dtype is f32 or bf16; weight gradients, LN
 *   statistics and the attention log-sum-exp are always f32.
 *
 * Ownership: the caller owns every device and host buffer it passes (device
 * arena, pinned host arena, parameters, gradients, x / y / dy / dx).  The
 * library keeps non-owning pointers and owns only HIP events and host
 * metadata.  Calls are asynchronous on the caller's streams; x, y, dy, dx
 * must stay valid until the compute stream has passed the call.
 *
 * Errors: every call returns TPS_OK (0) or a negative TPS_E* code and sets a
 * thread-local message readable with tps_last_error().  No C++ exception
 * crosses the ABI.  Asynchronous kernel and copy faults surface at
 * tps_stage_sync().
 */
#ifndef TPSTAGE_H
#define TPSTAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TPS_ABI_VERSION 7
#define TPS_MAX_MICRO 64

/* return codes */
enum {
  TPS_OK = 0,
  TPS_EINVAL = -1,   /* bad configuration or argument                        */
  TPS_ENOMEM = -2,   /* arena smaller than the plan needs                    */
  TPS_EORDER = -3,   /* call out of the planned F/B order, mb out of range   */
  TPS_EHIP = -4,     /* HIP runtime error (message in tps_last_error)        */
  TPS_ETIMEOUT = -5, /* a bounded wait expired                               */
  TPS_ESTATE = -6    /* call not valid in the stage's current state          */
};

/* storage dtypes */
enum { TPS_F32 = 0, TPS_BF16 = 1 };

/* per-tensor policy */
enum { TPS_KEEP = 0, TPS_RECOMPUTE = 1, TPS_OFFLOAD = 2 };

/* per-(layer, micro-batch) tensors read by the backward pass */
enum {
  TPS_T_X = 0,   /* layer input                         [T, h]            */
  TPS_T_A,       /* LN1 output                          [T, h]            */
  TPS_T_QKV,     /* packed projections                  [T, 3h]           */
  TPS_T_O,       /* attention output                    [T, h]            */
  TPS_T_LSE,     /* attention log-sum-exp, f32          [b, heads, seq]   */
  TPS_T_X1,      /* residual after attention            [T, h]            */
  TPS_T_C,       /* LN2 output                          [T, h]            */
  TPS_T_U,       /* FC1 pre-activation                  [T, f]            */
  TPS_T_G,       /* GeLU output                         [T, f]            */
  TPS_T_LN1,     /* LN1 mean and rstd, f32              [2, T]            */
  TPS_T_LN2,     /* LN2 mean and rstd, f32              [2, T]            */
  TPS_T_COUNT
};

/* weights placement */
enum { TPS_W_RESIDENT = 0, TPS_W_STREAM = 1 };

/* recompute granularity: LAYER replays one layer just before its backward
 * (layer-grouped); SEGMENT replays every recomputed tensor of the stage for
 * the micro-batch before its backward starts (block-wise T-Recomp). */
enum { TPS_GRAN_LAYER = 0, TPS_GRAN_SEGMENT = 1 };

/* format of the streamed parameter blocks in host memory (T-Offload's
 * weight reload): the storage dtype, or FP8 E4M3 codes with one f32 scale per
 * matrix row (the four weight matrices; vectors stay in the storage dtype),
 * expanded on the device to the storage dtype as bf16(decode(q) * scale). */
enum { TPS_Q_NONE = 0, TPS_Q_FP8_ROW = 1 };

/* where a layer backward's parameter-gradient kernels (weight-gradient GEMMs,
 * bias and LayerNorm column sums) run: SIDE forks them onto a stream of the
 * stage's own, beside the input-gradient chain on the compute stream; INLINE
 * issues them on the compute stream in the same order; AUTO picks INLINE when
 * a micro-batch has 4096 tokens or more (there every kernel of the chain fills
 * the chip, and two concurrent GEMMs slow each other more than the overlap
 * gains), else SIDE.  Results are bit-identical either way. */
enum { TPS_WGRAD_AUTO = 0, TPS_WGRAD_SIDE = 1, TPS_WGRAD_INLINE = 2 };

/* layer kind.  GPT: the pre-LN decoder layer above (LayerNorm, biases, GeLU
 * MLP, multi-head attention).  LLAMA: the LLAMA-style layer of the paper's
 * LLAMA2-70B workload (Section 6.1, "Workloads"; architecture from the public
 * LLAMA-2 description): RMSNorm (gains only, eps inside the root), no
 * biases, rotary position embedding of q and k (pairs (i, i + d/2) of each
 * head turned by pos * rope_base^(-2i/d)), grouped-query attention with
 * n_kv_heads key/value heads (query head n reads key/value head
 * n / (n_heads / n_kv_heads)), and a SwiGLU MLP g = SiLU(gate) * up with the
 * gate and up projections packed in one [2f, h] matrix (gate rows first).
 * LLAMA needs bf16 storage and head dim 128.  Tensor shapes under LLAMA:
 * QKV [T, (n_heads + 2 n_kv_heads) d] stored after the rotation, U [T, 2f]
 * (gate | up), G [T, f], LN1/LN2 [T] f32 (the reciprocal RMS); parameter
 * blocks hold W_QKV [(n_heads + 2 n_kv_heads) d, h], W_O, W_1 [2f, h], W_2,
 * G1, G2, and the bias / shift slots are empty (zero bytes). */
enum { TPS_ARCH_GPT = 0, TPS_ARCH_LLAMA = 1 };

/* op kinds in the planned order (TPS_OP_R: a recompute task of the T-Pipe
 * schedule, reported by tps_tpipe_schedule; a stage runs the recompute of a
 * micro-batch at the start of its backward) */
enum { TPS_OP_F = 0, TPS_OP_B = 1, TPS_OP_R = 2 };

/* parameter order inside one layer's packed parameter / gradient block */
enum {
  TPS_P_W_QKV = 0, TPS_P_B_QKV, TPS_P_W_O, TPS_P_B_O, TPS_P_W_1, TPS_P_B_1,
  TPS_P_W_2, TPS_P_B_2, TPS_P_G1, TPS_P_BE1, TPS_P_G2, TPS_P_BE2, TPS_P_COUNT
};

typedef struct tps_config {
  int32_t abi_version;          /* TPS_ABI_VERSION                              */
  int32_t n_layers;             /* L >= 1                                       */
  int32_t hidden;               /* h, multiple of 8                             */
  int32_t n_heads;              /* h / n_heads must be 64 or 128                */
  int32_t mlp;                  /* f, multiple of 8                             */
  int32_t seq;                  /* s >= 1 (any value)                           */
  int32_t micro_batch;          /* b >= 1                                       */
  int32_t n_micro;              /* M, 1..TPS_MAX_MICRO                          */
  int32_t dtype;                /* TPS_F32 or TPS_BF16                          */
  float ln_eps;                 /* LayerNorm epsilon (biased variance)          */
  const uint8_t* policy;        /* [n_layers][TPS_T_COUNT] TPS_KEEP/RECOMPUTE/OFFLOAD;
                                   NULL = keep everything.  X of layer 0 cannot
                                   be RECOMPUTE.  With TPS_GRAN_LAYER, X of every
                                   layer must be KEEP or OFFLOAD.               */
  uint64_t offload_mb_mask;     /* bit mb set: OFFLOAD entries apply to mb; for
                                   other micro-batches OFFLOAD acts as KEEP.    */
  int32_t offload_auto;         /* 1: ignore offload_mb_mask and pick victims
                                   by slack (see tps_plan)                     */
  int32_t weights;              /* TPS_W_RESIDENT or TPS_W_STREAM               */
  int32_t window;               /* streamed layers resident at once,
                                   2..max(2, n_layers)                          */
  int32_t recompute_granularity;/* TPS_GRAN_LAYER or TPS_GRAN_SEGMENT           */
  int32_t n_ops;                /* 0: default order from `inflight`             */
  const int32_t* ops;           /* n_ops pairs (TPS_OP_F|TPS_OP_B, mb)          */
  int32_t inflight;             /* default order: W forwards, then B(i), F(i+W)
                                   alternately, then the remaining backwards;
                                   0 means W = n_micro                          */
  float link_gbps_hint;         /* host-link GB/s per direction for victim choice */
  float tflops_hint;            /* sustained TFLOP/s for victim choice          */
  int32_t lookahead;            /* prefetch an offloaded mb this many ops before
                                   its backward (>= 1)                          */
  int32_t weights_quant;        /* TPS_Q_NONE, or TPS_Q_FP8_ROW (streamed bf16
                                   weights only): the host parameter blocks are
                                   in the quantized layout of
                                   tps_param_layout_q                           */
  int32_t wgrad_stream;         /* TPS_WGRAD_AUTO, _SIDE or _INLINE             */
  int32_t arch;                 /* TPS_ARCH_GPT or TPS_ARCH_LLAMA               */
  int32_t n_kv_heads;           /* LLAMA: key/value heads, dividing n_heads (0:
                                   n_heads); GPT: 0 or n_heads                  */
  float rope_base;              /* LLAMA: rotary base (0: 10000)                */
  int32_t group_wgrad;          /* 1: a backward group of several micro-batches
                                   at layer granularity issues each weight-
                                   gradient product once per layer over all of
                                   them (K = n T tokens) instead of once per
                                   micro-batch; the plan keeps the operands of
                                   the group's micro-batches for the layer
                                   (layers whose a, o, c, g are recomputed).
                                   Outputs are bit-identical; weight gradients
                                   equal the per-micro-batch sums up to the f32
                                   summation order.  0: per micro-batch.        */
} tps_config;

typedef struct tps_plan_info {
  uint64_t device_arena_bytes;  /* size of tps_memory.device_arena to allocate   */
  uint64_t host_arena_bytes;    /* size of the pinned host arena                 */
  uint64_t slot_bytes;          /* one micro-batch's resident checkpoints (KEEP) */
  int32_t n_slots;              /* resident checkpoint slots held at the peak    */
  uint64_t offload_slot_bytes;  /* one micro-batch's OFFLOAD tensors (device
                                   staging slot and host slot share the layout) */
  int32_t n_offload_slots;      /* device staging slots held at the peak         */
  int32_t n_host_slots;         /* pinned host slots held at the peak            */
  int32_t max_inflight;         /* micro-batches between F and B at the peak     */
  uint64_t replay_bytes;        /* recompute (replay) buffer                     */
  uint64_t work_bytes;          /* backward working buffers                      */
  uint64_t weight_window_bytes; /* streamed weight + grad window (STREAM)        */
  uint64_t param_bytes;         /* one layer's packed parameter block            */
  uint64_t grad_bytes;          /* one layer's packed f32 gradient block         */
  uint64_t keep_all_bytes;      /* activations if every tensor were kept, at the
                                   same in-flight peak (comparison)              */
  uint64_t predicted_peak_bytes;/* device arena + resident params + grads        */
  uint64_t offload_mb_mask;     /* effective mask (after auto selection)         */
  int32_t n_offload_mbs;
  int32_t n_replay_layers;      /* layers with at least one recomputed tensor    */
  double fwd_flops;             /* algorithmic flops per iteration               */
  double bwd_flops;
  double recompute_flops;       /* extra forward work the policy implies         */
  uint64_t h2d_bytes;           /* host-link traffic per iteration               */
  uint64_t d2h_bytes;
  int32_t wgrad_inline;         /* 1: parameter gradients on the compute stream */
  int32_t group_wgrad_slots;    /* micro-batches a backward group can batch its
                                   weight gradients over (0: not batched)       */
} tps_plan_info;

typedef struct tps_params {
  /* [n_layers] pointers to packed parameter blocks in storage dtype, laid out
   * by tps_param_layout().  RESIDENT: device pointers.  STREAM: pinned host
   * pointers (the library streams them in). */
  void* const* layer_params;
  /* [n_layers] pointers to packed f32 gradient blocks (same order, f32).
   * RESIDENT: device pointers.  STREAM: pinned host pointers. */
  float* const* layer_grads;
} tps_params;

typedef struct tps_memory {
  void* device_arena;           /* >= plan.device_arena_bytes, 256-byte aligned */
  uint64_t device_bytes;
  void* host_arena;             /* pinned, >= plan.host_arena_bytes (may be NULL
                                   when that is 0)                              */
  uint64_t host_bytes;
  void* compute_stream;         /* hipStream_t for kernels (NULL: the null
                                   stream); the stage forks the backward's
                                   parameter-gradient kernels (and light
                                   segment replays) onto streams of its own
                                   and joins them back before anything on this
                                   stream reads their results, and at the end
                                   of each forward and of the iteration       */
  void* copy_stream;            /* hipStream_t for device -> host copies, or
                                   NULL: the stage creates its own             */
  void* prefetch_stream;        /* hipStream_t for host -> device copies, or
                                   NULL: the stage creates its own; the same
                                   stream as copy_stream puts both directions
                                   on one stream.  Separate streams let both
                                   link directions run at once (the offloads of
                                   later micro-batches under the prefetches of
                                   earlier ones, Section 5).  Streams the stage
                                   creates each hold a hardware queue that no
                                   other stream shares (a stream sharing a
                                   queue with a copy stream waits behind its
                                   copies) and synchronize with the null
                                   stream.  Copy streams are used, and created,
                                   only when the plan moves data over the host
                                   link; a caller's copy stream must differ
                                   from compute_stream                         */
} tps_memory;

typedef struct tps_stats {
  uint64_t h2d_bytes, d2h_bytes;/* issued this iteration                        */
  uint64_t kernels;             /* kernel launches this iteration               */
  uint64_t replays;             /* recompute replays (layers) this iteration    */
  int32_t ops_done;             /* position in the planned order                */
  double host_update_ms;        /* host optimizer: summed duration of the layer
                                   updates finished since the iteration began   */
  double host_wait_ms;          /* time the issuing thread waited for a layer's
                                   update before reloading it, this iteration   */
  int32_t host_updates;         /* layer updates finished since it began        */
} tps_stats;

typedef struct tps_kernel_time {
  char name[120];               /* kernel (or fixed kernel sequence) name       */
  uint64_t launches;
  double ms;                    /* summed durations between HIP events recorded
                                   on the compute stream around each launch     */
  double flops;                 /* summed algorithmic flops                     */
  double bytes;                 /* summed algorithmic HBM bytes                 */
} tps_kernel_time;

typedef struct tps_stage tps_stage;

/* Layout of one layer's packed parameter block (storage dtype) and gradient
 * block (f32): byte offsets of the TPS_P_COUNT tensors, each 256-byte aligned.
 * Shapes: W_qkv[3h,h] b_qkv[3h] W_o[h,h] b_o[h] W_1[f,h] b_1[f] W_2[h,f] b_2[h]
 * g1[h] be1[h] g2[h] be2[h]. */
int tps_param_layout(const tps_config* cfg, uint64_t param_offsets[TPS_P_COUNT],
                     uint64_t* param_bytes, uint64_t grad_offsets[TPS_P_COUNT],
                     uint64_t* grad_bytes);

/* Layout of one layer's quantized host parameter block (TPS_Q_FP8_ROW):
 * byte offsets of the TPS_P_COUNT tensors (uint8 E4M3 codes [rows][cols] for
 * W_qkv, W_o, W_1, W_2; storage dtype for the vectors) and of the f32 row
 * scales of the four matrices (in the order W_qkv, W_o, W_1, W_2), each
 * 256-byte aligned, and the block size. */
int tps_param_layout_q(const tps_config* cfg, uint64_t offsets[TPS_P_COUNT], uint64_t scale_offsets[4],
                       uint64_t* bytes);

/* Host only, no GPU needed.  Validates the config, resolves the op order and
 * the policy closure, assigns checkpoint slots over the order, lays out the
 * arenas and predicts the peak.  With offload_auto, victims are picked in
 * decreasing order of slack between F(mb) and B(mb) (the poorest temporal
 * locality first, Section 3 and Section 4.2) while the simulated round trip
 * at link_gbps_hint stays hidden behind compute at tflops_hint. */
int tps_plan(const tps_config* cfg, tps_plan_info* out);

/* Create a stage.  Copies the config and policy; keeps the pointers of
 * params and mem.  Launches nothing.
 * Debug: with the environment variable TPS_POISON set (and not "0") when the
 * stage is created, memory whose contents are dead by the stage's protocol is
 * filled with all-ones bytes (NaN in f32 and bf16) as it is handed back: a
 * staging slot after its copy to host or its micro-batch's backward, the
 * checkpoint slot and the replay buffer after each backward, the transposed
 * weights of an evicted window entry.  Results are unchanged unless a read
 * escapes the protocol; each fill costs one kernel. */
int tps_stage_init(const tps_config* cfg, const tps_params* params,
                   const tps_memory* mem, tps_stage** out);

/* Start an iteration: resets the order cursor; zero_grads != 0 restarts the
 * gradients from zero: with resident weights the iteration's first backward
 * contribution to each gradient tensor writes it instead of adding to it (the
 * bytes between tensors in a block are left as they are), with streamed
 * weights the host blocks are cleared as each layer is first used.
 * Parameters may change between iterations (an optimizer step): resident
 * weights get their transposed copies rebuilt here, and streamed weights are
 * brought in again from the host blocks for every layer (no layer runs on a
 * copy made in an earlier iteration).  With streamed weights the caller
 * changes the pinned host blocks, or reads the host gradient blocks, only
 * after tps_stage_sync() has followed the iteration's last op. */
int tps_stage_begin_iteration(tps_stage* st, int zero_grads);

/* F(mb): x, y are [b, s, h] device buffers in storage dtype. */
int tps_stage_forward(tps_stage* st, int mb, const void* x, void* y);

/* B(mb): dy, dx are [b, s, h] device buffers in storage dtype.  Adds the
 * micro-batch's parameter gradients into the f32 gradient blocks. */
int tps_stage_backward(tps_stage* st, int mb, const void* dy, void* dx);

/* Layer-major groups: F(mb0..mb0+n-1) (resp. B) run layer by layer, so a
 * streamed layer is brought in once for the whole group.  x[i], y[i] (resp.
 * dy[i], dx[i]) belong to micro-batch mb0 + i. */
int tps_stage_forward_group(tps_stage* st, int mb0, int n, const void* const* x,
                            void* const* y);
int tps_stage_backward_group(tps_stage* st, int mb0, int n, const void* const* dy,
                             void* const* dx);

/* Wait for every stream of the stage (compute, parameter-gradient, replay
 * and copy streams); reports asynchronous faults as TPS_EHIP. */
int tps_stage_sync(tps_stage* st);

/* The same wait with a deadline: returns TPS_OK once every stream of the
 * stage is idle, TPS_EHIP if a stream reports a fault, and TPS_ETIMEOUT
 * (naming a busy stream) if work is still pending after timeout_ms
 * milliseconds (0 = just test).  A timeout leaves the work running: the
 * stage stays usable and a later sync completes it.  TPS_EINVAL for a
 * negative timeout. */
int tps_stage_sync_for(tps_stage* st, double timeout_ms);

int tps_stage_stats(const tps_stage* st, tps_stats* out);

/* Measurement: from now on bracket every launch whose kernel name starts
 * with `prefix` with HIP timing events on the compute stream ("" times every
 * kernel, NULL turns timing off), and clear the accumulated times.  Single-
 * kernel launches carry the demangled kernel name a profiler prints; fixed
 * multi-kernel sequences (attention backward, LayerNorm backward, column
 * sums) carry one name for the sequence. */
int tps_stage_time_kernels(tps_stage* st, const char* prefix);

/* Waits for the compute stream, then reports per-name totals accumulated
 * since the last tps_stage_time_kernels(); writes at most `max` entries and
 * the number of names to *n_out. */
int tps_stage_kernel_times(tps_stage* st, tps_kernel_time* out, int max, int* n_out);

/* Releases events and host metadata (caller buffers are untouched). */
int tps_stage_destroy(tps_stage* st);

/* Pinned (page-locked) host memory of exactly `bytes` bytes, for the host
 * side of streamed weights and gradients and for the host arena: T-Offload
 * moves these between host DRAM and HBM with asynchronous copies (Section 5),
 * which need page-locked memory.  *out receives the pointer (NULL when bytes
 * is 0); the caller releases it with tps_host_free.  TPS_ENOMEM when the
 * system cannot pin that much. */
int tps_host_alloc(uint64_t bytes, void** out);
int tps_host_free(void* p);

/* T-Pipe two-chunk pipeline schedule and unit-time simulator (host only, no
 * GPU needed).  Paper: Section 4.1 "T-Pipe Schedule" and the appendix
 * "Theoretical Analysis of T-Pipe" (two chunks per stage, chunk 1 the
 * shallow layer block s, chunk 2 the deep block p + s; forward 1 T_unit and
 * backward 2 T_unit per chunk and stage); Section 4.2 "Addressing the
 * Concerns" and the appendices on the delay rounds and on T-Recomp
 * (block-wise recompute of chunk 1 as a task of its own, 1 T_unit, before
 * that chunk's backward; chunk 2 delayed by k rounds).
 *
 * Each stage runs its tasks in the T-Pipe order (rounds of F chunk 1,
 * B chunk 2, F chunk 2, B chunk 1); the simulator starts every task as soon
 * as its stage is free and its dependencies have finished.  Activation
 * blocks (m_a / 2p each) are held from the start of a chunk's forward to the
 * start of its backward on the stage; a recomputed chunk holds none and its
 * regenerated activations take one buffer block from the recompute to the
 * end of the backward. */
typedef struct tps_tpipe_config {
  int32_t stages;               /* p, 1..256                                    */
  int32_t micro;                /* m micro-batches per mini-batch, 1..4096      */
  int32_t t_recomp;             /* 1: block-wise T-Recomp of chunk 1            */
  int32_t delay;                /* chunk-2 delay rounds k, or -1: the smallest k
                                   that reaches the shortest makespan          */
} tps_tpipe_config;

typedef struct tps_tpipe_task {
  int32_t kind;                 /* TPS_OP_F, TPS_OP_B or TPS_OP_R               */
  int32_t chunk;                /* 1 (shallow) or 2 (deep)                      */
  int32_t mb;                   /* micro-batch                                  */
  int32_t start, end;           /* simulated time, T_unit                       */
} tps_tpipe_task;

typedef struct tps_tpipe_result {
  int32_t delay;                /* k used                                       */
  int32_t makespan;             /* whole pipeline, T_unit                       */
  int32_t busy;                 /* busy time of one stage, T_unit               */
  double bubble_ratio;          /* (makespan - busy) / makespan                 */
  int32_t peak_blocks_chunk1;   /* at the requested stage, blocks of m_a / 2p   */
  int32_t peak_blocks_chunk2;
  int32_t peak_buffer_blocks;   /* recompute buffer (T-Recomp)                  */
  int32_t peak_blocks;          /* all three together at the requested stage   */
  int32_t max_stage_peak_blocks;/* the largest peak_blocks over all stages      */
  int32_t life_chunk1;          /* start of forward to start of backward of the
                                   middle micro-batch on the requested stage   */
  int32_t life_chunk2;
  int32_t offload_window;       /* idle time of the requested stage from the end
                                   of chunk 2's last backward to the start of
                                   chunk 1's last backward (room for chunk 2's
                                   gradient offload and host optimizer step)  */
  int32_t upload_window;        /* idle time of the requested stage from its
                                   first task to chunk 2's first forward (room
                                   for the reload of chunk 2's weights)        */
} tps_tpipe_result;

/* Simulates the schedule and writes the requested stage's tasks in execution
 * order (at most max_tasks of them; *n_tasks receives the count: 4m, or 5m
 * with T-Recomp) and the summary.  Splitting the list by chunk gives the F/B
 * order of each chunk's layers (tps_config.ops, recompute tasks folded into
 * the backward that follows them).  TPS_EINVAL for out-of-range arguments. */
int tps_tpipe_schedule(const tps_tpipe_config* cfg, int32_t stage, tps_tpipe_task* tasks,
                       int32_t max_tasks, int32_t* n_tasks, tps_tpipe_result* out);

/* AdamW hyper-parameters of the host optimizer update. */
typedef struct tps_adamw {
  float lr;                     /* learning rate (>= 0)                         */
  float beta1, beta2;           /* moment decay rates in [0, 1)                 */
  float eps;                    /* added to sqrt of the second moment (>= 0)    */
  float weight_decay;           /* decoupled weight decay (>= 0)                */
} tps_adamw;

/* T-Offload's host-side model-state update of one layer (paper, Section 5:
 * gradients offloaded after the layer's last backward, optimizer update on
 * the CPU, weights reloaded in quantized form).  All arrays are host memory:
 * master, m, v and grad are f32 in the layout of the layer's gradient block
 * (tps_param_layout's gradient offsets).  With step >= 1 one AdamW step is
 * applied in place to master, m and v:
 *   m = b1 m + (1 - b1) g,  v = b2 v + (1 - b2) g^2,
 *   w = w - lr (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps) - lr wd w;
 * with step == 0 nothing is updated (m, v, grad and opt may be NULL).  Then
 * params_out receives the layer's parameter block as the device will load
 * it: quant == TPS_Q_NONE in the storage dtype (tps_param_layout, bf16
 * rounded to nearest even), TPS_Q_FP8_ROW in the quantized layout of
 * tps_param_layout_q (matrix rows as E4M3 codes of w / scale with
 * scale = max|row| / 448 in f32, nearest code, ties to an even mantissa,
 * saturating at 448; vectors in bf16).  Runs on n_threads host threads
 * (0: one per hardware thread) and returns when done.  TPS_EINVAL for bad
 * arguments. */
int tps_host_adamw_layer(const tps_config* cfg, const tps_adamw* opt, int32_t step, float* master, float* m,
                         float* v, const float* grad, void* params_out, int32_t quant, int32_t n_threads);

/* Turns on the model-state half of T-Offload for a stage with streamed
 * weights (paper, Section 5): in every iteration, once all backwards have
 * passed layer l, its f32 gradient block goes to the host and a host thread
 * of the stage applies one AdamW step (tps_host_adamw_layer semantics, step
 * numbers first_step, first_step + 1, ... per layer, n_threads threads) to
 * the layer's master weights and moments and rewrites the layer's pinned
 * parameter block (storage dtype, or the quantized layout when the config
 * has weights_quant); the update overlaps the backward of the layers below,
 * and the layer's next load waits for it.  master, m, v: [n_layers] pinned or
 * pageable host f32 blocks in the gradient-block layout (master initialised
 * to the weights, m and v to zero), owned by the caller and not touched by
 * the caller while updates may run (until tps_stage_sync returns, which also
 * waits for the updates and reports their errors).  Call between iterations;
 * iterations should start with zero_grads set.  TPS_EINVAL without streamed
 * weights or with bad arguments, TPS_ESTATE if already set. */
int tps_stage_set_optimizer(tps_stage* st, const tps_adamw* opt, float* const* master, float* const* m,
                            float* const* v, int32_t first_step, int32_t n_threads);

/* As tps_stage_set_optimizer, with the model state of the shallowest
 * n_device layers (0 .. n_device - 1) kept on the GPU (paper, Section 5 and
 * the T-Offload scalability appendix: the shallow chunk's states stay on the
 * device where no bubble hides their offload; on one GPU layer 0's update
 * would otherwise sit between two iterations).  For those layers master[l],
 * m[l] and v[l] are device f32 blocks (gradient-block layout, 16-byte
 * aligned) and dparams[l] a device parameter block in the storage dtype
 * (tps_param_layout) holding the layer's current parameters, all owned by the
 * caller.  Once every backward of an iteration has passed such a layer, its
 * AdamW step runs on the compute stream with the host update's arithmetic
 * (the same f32 operations, hence the same bits), writing master, m, v and
 * dparams[l]; its final gradients are consumed on the device (its host
 * gradient block is no result: it holds at most partial sums from times the
 * layer left the window during the iteration), and its loads copy dparams[l]
 * (its pinned host parameter block is no longer read, and with weights_quant
 * its parameters are not quantized).
 * Iterations must start with zero_grads set.  n_device in 0 .. n_layers
 * (dparams may be NULL when 0); TPS_EINVAL otherwise, or for a null or
 * misaligned device block. */
int tps_stage_set_optimizer_split(tps_stage* st, const tps_adamw* opt, float* const* master, float* const* m,
                                  float* const* v, void* const* dparams, int32_t n_device, int32_t first_step,
                                  int32_t n_threads);

/* Thread-local message of the last failing call ("" if none). */
const char* tps_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TPSTAGE_H */
