// Stage executor: runs F(mb) and B(mb) in the planned order on the caller's
// compute stream (the backward's parameter-gradient kernels on a stream of
// its own, light segment replays of lower layers on another), with
//  - the recompute engine: the replay program of each layer re-runs the same
//    forward kernels with the same launch shapes, so regenerated tensors are
//    bit-identical to the ones the forward produced; SEGMENT granularity
//    replays every layer of the micro-batch before its backward starts
//    (block-wise T-Recomp), LAYER granularity replays one layer just before
//    that layer's backward;
//  - the offload engine: OFFLOAD tensors of offloaded micro-batches go to
//    pinned host slots on the copy stream after each layer's forward and come
//    back `lookahead` ops before the backward; cross-stream hazards on the
//    staging slots are ordered by events recorded at every release and waited
//    on at every acquire;
//  - streamed weights: a window of layer parameter blocks (and f32 gradient
//    blocks) in the arena, brought in on the copy stream ahead of use.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <chrono>
#include <condition_variable>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <map>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "errors.h"
#include "kernels.h"
#include "planner.h"

using namespace tps;

namespace {

#define TPS_HIP(expr)                                      \
  do {                                                     \
    hipError_t _e = (expr);                                \
    if (_e != hipSuccess) return check_hip(_e, #expr);     \
  } while (0)

#define TPS_TRY(expr)              \
  do {                             \
    int _rc = (expr);              \
    if (_rc != TPS_OK) return _rc; \
  } while (0)

// A stream the stage owns, on a hardware queue that no other stream shares.
// The runtime multiplexes ordinary streams over a small pool of hardware
// queues (GPU_MAX_HW_QUEUES, four by default, the default stream among
// them); two streams on one queue run in submission order, so a kernel stream
// that lands on the queue of a copy stream stalls behind every barrier the
// copies put there.  A stream created with a CU mask gets a queue of its own
// from the ROCm runtime; the mask here enables every CU.  Such streams are
// blocking streams: they synchronize with the null stream.
hipError_t queue_stream(int device, hipStream_t* s) {
  int ncu = 0;
  hipError_t e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess) return e;
  std::vector<uint32_t> mask((size_t)(ncu + 31) / 32, 0xFFFFFFFFu);
  return hipExtStreamCreateWithCUMask(s, (uint32_t)mask.size(), mask.data());
}

// Device-to-host copy issued as a pitched (2D) copy of 4 MiB rows plus one
// row for the remainder.  With the framework's runtime initialised first, a
// plain device-to-host copy runs as a copy kernel on every CU for its whole
// duration (tens of milliseconds per gradient block, beside the GEMMs); the
// pitched form runs on the copy engines.
hipError_t d2h_async(void* dst, const void* src, size_t bytes, hipStream_t s) {
  constexpr size_t W = size_t(4) << 20;
  const size_t rows = bytes / W, tail = bytes - rows * W;
  if (rows) {
    const hipError_t e = hipMemcpy2DAsync(dst, W, src, W, W, rows, hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return e;
  }
  if (tail)
    return hipMemcpy2DAsync(static_cast<char*>(dst) + rows * W, tail, static_cast<const char*>(src) + rows * W, tail,
                            tail, 1, hipMemcpyDeviceToHost, s);
  return hipSuccess;
}

// Products with a long contraction take the weight operand in its [K][N]
// form (NN layout): each tile load instruction then covers two 512-byte row
// segments instead of eight 128-byte ones.  On MI355X that was 6-20% faster
// for K >= 12288 (hidden 5120-8192 MLP and QKV shapes) and up to 10% slower
// for shorter K, where the [N][K] form (NT) stays.
bool nn_for(int K) { return K >= 12288; }

struct SlotEvent {
  hipEvent_t ev = nullptr;
  bool valid = false;
};

// Streamed-weight window entry.
struct WinEntry {
  int layer = -1;
  bool grads_live = false;     // the device grad block holds this layer's sums
  SlotEvent param_ready;       // H2D of the parameters finished (copy stream)
  SlotEvent last_use;          // last kernel reading the entry (compute stream)
  SlotEvent grads_out;         // D2H of the grads finished (copy stream)
  bool wt_valid = false;       // transposed copies match the parameters
  uint64_t tick = 0;
};

}  // namespace

struct tps_stage {
  Plan p;
  std::vector<char*> lp;     // per-layer parameter block (device, or pinned host when streamed)
  std::vector<float*> lg;    // per-layer f32 gradient block (device, or pinned host when streamed)
  char* arena = nullptr;
  bool bpart_clean = false;   // the bias partial blocks are all zero (no layer backward cut short)
  char* host = nullptr;
  // cs: kernels; xs: device -> host copies; ps: host -> device copies (the
  // caller's, or the stage's own when it gives none: own_xs, own_ps)
  hipStream_t cs = nullptr, xs = nullptr, ps = nullptr;
  bool own_xs = false, own_ps = false;
  // gs: the layer backward's parameter-gradient kernels (weight GEMMs, column
  // sums, finalize), forked from cs where their inputs are ready and joined
  // back at the end of the layer (gs is cs itself when the plan issues them
  // inline: the forks and joins are then no-ops); ks: the stream the next
  // kernel goes to
  hipStream_t gs = nullptr, ks = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  // deferred joins: layer backwards of an iteration are numbered in issue
  // order (bstep); ev_gs[k] marks the end of the last parameter-gradient work
  // of a layer backward with bstep parity k (layer gs_layer[k]), which read
  // the buffers of set k; gs_pending[k]: cs has not waited for it yet
  hipEvent_t ev_gs[2] = {nullptr, nullptr};
  bool gs_pending[2] = {false, false};
  int gs_layer[2] = {-1, -1};
  int bstep = 0;
  // grads_fresh[l]: layer l's gradient block counts as zero (requested by
  // begin_iteration, or a streamed layer's first load for a backward of the
  // iteration, and not yet written): its next layer backward writes the
  // gradients instead of adding to them, so no zero fill is needed
  std::vector<char> grads_fresh;
  // rs: replays of all but the first replayed layer of a segment run here,
  // beside the backward chain on cs (lagging configuration with light,
  // independent layer replays only); ev_replay[l] marks layer l's replay done
  hipStream_t rs = nullptr;
  hipEvent_t ev_rfork = nullptr;
  std::vector<hipEvent_t> ev_replay;
  std::vector<char> replay_on_rs;
  int device = 0;

  std::vector<SlotEvent> oslot_ev;               // last release of each offload slot
  std::vector<SlotEvent> offloaded_ev;           // [M] last device -> host copy of the mb issued (xs)
  std::vector<SlotEvent> hslot_read_ev;          // [host slots] last prefetch out of the slot (ps)
  std::vector<SlotEvent> lgrads_out_ev;          // [L] last flush of the layer's grads to host (xs)
  std::vector<std::vector<hipEvent_t>> ready_ev; // [M][L] H2D of (mb, layer) done
  std::vector<char> prefetched;
  hipEvent_t ev_tmp = nullptr;

  // streamed weights
  std::vector<WinEntry> win;
  std::vector<char> grads_touched;  // [L] this iteration
  uint64_t tick = 0;

  // T-Offload of model state: the host optimizer update of each layer, run
  // by a worker thread once the layer's final gradients of the iteration are
  // on the host; the layer's next load waits for it
  struct HostOpt {
    bool on = false;
    tps_adamw hp{};
    int threads = 0;
    std::vector<float*> master, m, v;
    std::vector<int> step;           // step number of the layer's next update
    std::vector<int> bpass;          // layer backwards this iteration
    std::vector<hipEvent_t> final_ev;   // final gradient flush of the layer (copy stream)
    std::vector<char> pending;       // update queued or running
    // layers 0 .. n_dev - 1 are updated on the device: master, m, v are device
    // blocks, dparams[l] the layer's device parameter block (loads copy it),
    // dev_ev[l] the end of its last update (compute stream)
    int n_dev = 0;
    std::vector<void*> dparams;
    std::vector<hipEvent_t> dev_ev;
    std::vector<char> dev_ev_valid;
    std::deque<int> queue;
    std::mutex mu;
    std::condition_variable cv;
    std::thread worker;
    bool stop = false;
    int rc = TPS_OK;
    std::string err;
  } hopt;
  int opt_after_backward(int l, int passes);
  int wait_layer_update(int l);
  int wait_all_updates();
  void opt_worker();

  // kernel timing (measurement only)
  struct TimedLaunch {
    std::string name;
    double flops, bytes;
    hipEvent_t a, b;
    hipStream_t on;
  };
  bool timing = false;
  std::string tprefix;
  std::vector<TimedLaunch> tpending;
  std::vector<hipEvent_t> tpool;
  std::map<std::string, tps_kernel_time> tagg;
  int kbegin(const char* name, double flops, double bytes);
  int kend(int idx);
  int kresolve();

  int cursor = 0;
  std::vector<char> f_done, b_done;
  bool in_iteration = false;
  tps_stats stats{};

  // --- pointers -----------------------------------------------------------
  char* kslot_base(int mb) const { return arena + p.off_kslots + (uint64_t)p.kslot[mb] * p.kslot_bytes; }
  char* oslot_base(int slot) const { return arena + p.off_oslots + (uint64_t)slot * p.oslot_bytes; }
  char* host_base(int mb) const { return host + (uint64_t)p.host_slot[mb] * p.oslot_bytes; }

  // batched weight gradients of a backward group: while grp_i >= 0 the
  // recomputed a, o, c, g of the layer live in micro-batch slot grp_i of the
  // group's operand buffers (they are read again after the group's last
  // micro-batch)
  int grp_i = -1;
  static int grp_act_index(int t) {
    return t == TPS_T_A ? 0 : t == TPS_T_O ? 1 : t == TPS_T_C ? 2 : t == TPS_T_G ? 3 : -1;
  }
  char* grp_slot(uint64_t off, uint64_t slot_bytes, int i) const {
    return arena + p.off_work + off + (uint64_t)i * ((slot_bytes + 255) & ~uint64_t(255));
  }
  // device address of tensor t of (layer l, mb) for the phase (fwd or bwd)
  void* tensor(int l, int t, int mb, bool bwd) const {
    const size_t k = (size_t)l * TPS_T_COUNT + t;
    if (grp_i >= 0 && bwd && p.policy[k] == TPS_RECOMPUTE) {
      const int a = grp_act_index(t);
      if (a >= 0) return grp_slot(p.work.grp_act[a], p.tbytes[t], grp_i);
    }
    switch (p.policy[k]) {
      case TPS_RECOMPUTE: return arena + p.off_replay + p.replay_off[k];
      case TPS_KEEP: return kslot_base(mb) + p.kslot_off[k];
      default: return oslot_base(bwd ? p.oslot_b[mb] : p.oslot_f[mb]) + p.oslot_off[k];
    }
  }
  char* work(uint64_t off) const { return arena + p.off_work + off; }
  float* bpart(int l) const { return reinterpret_cast<float*>(arena + p.off_bpart + (uint64_t)l * p.bpart_bytes); }

  // --- events ---------------------------------------------------------------
  // TPS_POISON: memory whose contents the protocol declares dead (a staging
  // slot handed back, a checkpoint slot and the replay buffer after the
  // micro-batch's backward, the transposed weights of an evicted window
  // entry) is filled with all-ones bytes, a NaN in f32 and bf16, so a read
  // that should not happen shows in the results
  bool poison = false;
  bool llama_tables = false;   // rotation table and zero bias written
  int poison_fill(void* ptr, uint64_t bytes, hipStream_t on) {
    if (poison && bytes) TPS_HIP(fill_bytes_launch(ptr, bytes, 0xFF, on));
    return TPS_OK;
  }
  // after the backward of micro-batch mb: its checkpoint slot and the replay
  // buffer, once the parameter-gradient kernels that read them are done
  int poison_after_backward(int mb) {
    if (!poison) return TPS_OK;
    TPS_TRY(join_if_pending());
    if (p.kslot_bytes) TPS_TRY(poison_fill(kslot_base(mb), p.kslot_bytes, cs));
    TPS_TRY(poison_fill(arena + p.off_replay, p.replay_bytes, cs));
    return TPS_OK;
  }
  int release_oslot(int slot, hipStream_t on) {
    TPS_TRY(poison_fill(oslot_base(slot), p.oslot_bytes, on));
    TPS_HIP(hipEventRecord(oslot_ev[slot].ev, on));
    oslot_ev[slot].valid = true;
    return TPS_OK;
  }
  int acquire_oslot(int slot, hipStream_t on) {
    if (oslot_ev[slot].valid) TPS_HIP(hipStreamWaitEvent(on, oslot_ev[slot].ev, 0));
    return TPS_OK;
  }

  // --- parameters (resident or streamed window) ------------------------------
  const char* params_of(int l, int* entry);
  float* grads_of(int l, int entry);
  uint64_t entry_bytes() const { return p.pbytes + p.gbytes + (p.quant ? ((p.qbytes + 255) & ~uint64_t(255)) : 0); }
  char* qstage_of(int entry);
  int load_params(int l, int entry);
  char* wt_of(int l, int entry) const {
    return arena + p.off_wt + (uint64_t)(p.weights == TPS_W_STREAM ? entry : l) * p.wt_bytes;
  }
  int refresh_wt(int l, int entry);
  int ensure_layer(int l, bool for_backward, int* entry);
  int touch(int entry);
  int invalidate_window();
  int prefetch_layer(int l);
  int flush_grads(int entry);
  int flush_all_grads();
  int finalize_bias_grads(int l, float* G, bool overwrite);

  // --- compute ----------------------------------------------------------------
  int gemm(int layout, int epi, int M, int N, int K, const void* A, int64_t lda, const void* B, int64_t ldb,
           void* C, int64_t ldc, const void* bias = nullptr, const void* resid = nullptr, int64_t ldr = 0,
           void* aux = nullptr, int64_t ldaux = 0, bool overwrite = false) {
    ++stats.kernels;
    const double es = p.esize;
    const double bytes = ((double)M * K + (double)N * K) * es +
                         (epi == TPS_EPI_ACC_F32 ? (overwrite ? 4.0 : 8.0) * M * N : (double)M * N * es);
    const GemmArgs ga{M, N, K, A, lda, B, ldb, C, ldc, bias, resid, ldr, aux, ldaux, epi, 0, 0, overwrite};
    const int t = kbegin(gemm_kernel_name(p.dtype, layout, ga), 2.0 * M * N * K, bytes);
    const int rc = check_hip(gemm_launch(p.dtype, layout, epi, M, N, K, A, lda, B, ldb, C, ldc, bias, resid, ldr,
                                         aux, ldaux, ks, overwrite),
                             "gemm");
    return rc ? rc : kend(t);
  }
  const char* tname(const char* bf16_name, const char* f32_name) const {
    return p.dtype == TPS_BF16 ? bf16_name : f32_name;
  }
  int fwd_layer(int l, int mb, const char* W, void* y, uint32_t ops, bool replay, bool bwd_slots);
  // grp >= 0: micro-batch slot of a backward group whose weight gradients
  // are issued once per layer (batched_wgrad); the layer's gradient operands
  // go to the group's slots and the weight-gradient GEMMs are left out
  int bwd_layer(int l, int mb, const char* W, const char* WT, float* G, const void* dy, void* dx, int wp, bool defer,
                int grp = -1);
  int bwd_layer_llama(int l, int mb, const char* W, const char* WT, float* G, const void* dy, void* dx, int wp,
                      bool defer, int grp);
  bool layer_batchable(int l) const {
    for (int t : {TPS_T_A, TPS_T_O, TPS_T_C, TPS_T_G})
      if (p.pol(l, t) != TPS_RECOMPUTE) return false;
    return true;
  }
  int batched_wgrad(int l, float* G, int n, bool fresh, int yin);
  // stream `on` waits for the lagging parameter-gradient kernels of layer l
  // (and all gs work before them), if any are pending
  int wait_gs_layer_on(int l, hipStream_t on) {
    for (int k = 0; k < 2; ++k)
      if (gs_pending[k] && gs_layer[k] == l) TPS_HIP(hipStreamWaitEvent(on, ev_gs[k], 0));
    return TPS_OK;
  }
  // cs waits for the lagging parameter-gradient kernels of layer l (and all
  // gs work before them), if any are pending
  int wait_gs_layer(int l) {
    for (int k = 0; k < 2; ++k)
      if (gs_pending[k] && gs_layer[k] == l) {
        TPS_HIP(hipStreamWaitEvent(cs, ev_gs[k], 0));
        gs_pending[k] = false;
      }
    return TPS_OK;
  }
  int join_if_pending() { return (gs_pending[0] || gs_pending[1]) ? join_gs() : TPS_OK; }
  // cs waits for everything issued to gs so far
  int join_gs() {
    TPS_HIP(hipEventRecord(ev_join, gs));
    TPS_HIP(hipStreamWaitEvent(cs, ev_join, 0));
    gs_pending[0] = gs_pending[1] = false;
    return TPS_OK;
  }
  int forward_one(int mb, const void* x, void* y);
  int backward_one(int mb, const void* dy, void* dx);
  int prefetch_mb(int mb);
  int run_prefetches(int pos);
  int d2h_layer(int l, int mb);
  int check_op(int kind, int mb);
};

// ---------------------------------------------------------------------------
// Streamed weights.  Window entries hold a layer's parameter block and its
// f32 gradient block.  Eviction waits (on the copy stream) for the entry's
// last compute use; gradients leave with a D2H into the caller's host block
// and come back with an H2D if the layer is touched again in the iteration.
// ---------------------------------------------------------------------------
const char* tps_stage::params_of(int l, int* entry) {
  if (p.weights == TPS_W_RESIDENT) return lp[l];
  return arena + p.off_wwin + (uint64_t)(*entry) * entry_bytes();
}

float* tps_stage::grads_of(int l, int entry) {
  if (p.weights == TPS_W_RESIDENT) return lg[l];
  return reinterpret_cast<float*>(arena + p.off_wwin + (uint64_t)entry * entry_bytes() + p.pbytes);
}

// Staging area of a window entry for a quantized parameter block.
char* tps_stage::qstage_of(int entry) {
  return arena + p.off_wwin + (uint64_t)entry * entry_bytes() + p.pbytes + p.gbytes;
}

// Brings layer l's parameter block from its host block into window entry e on
// the prefetch stream: a plain copy, or the quantized block into the entry's
// staging area followed by its expansion to the storage dtype (matrices from
// E4M3 codes and row scales, vectors copied as they are).
int tps_stage::load_params(int l, int e) {
  int ent = e;
  char* dst = const_cast<char*>(params_of(l, &ent));
  if (hopt.on && l < hopt.n_dev) {
    // a layer updated on the device: its parameters in the storage dtype,
    // after its last update, or before the first one after the caller's
    // writes (which every call orders before the compute stream's work)
    if (hopt.dev_ev_valid[l]) {
      TPS_HIP(hipStreamWaitEvent(ps, hopt.dev_ev[l], 0));
    } else {
      TPS_HIP(hipEventRecord(ev_tmp, cs));
      TPS_HIP(hipStreamWaitEvent(ps, ev_tmp, 0));
    }
    TPS_HIP(hipMemcpyAsync(dst, hopt.dparams[l], p.pbytes, hipMemcpyDeviceToDevice, ps));
    return TPS_OK;
  }
  if (p.quant != TPS_Q_FP8_ROW) {
    TPS_HIP(hipMemcpyAsync(dst, lp[l], p.pbytes, hipMemcpyHostToDevice, ps));
    stats.h2d_bytes += p.pbytes;
    return TPS_OK;
  }
  char* q = qstage_of(e);
  TPS_HIP(hipMemcpyAsync(q, lp[l], p.qbytes, hipMemcpyHostToDevice, ps));
  stats.h2d_bytes += p.qbytes;
  const int mats[4] = {TPS_P_W_QKV, TPS_P_W_O, TPS_P_W_1, TPS_P_W_2};
  for (int k = 0; k < 4; ++k) {
    TPS_HIP(dequant_fp8_rows_launch(q + p.qoff[mats[k]], reinterpret_cast<const float*>(q + p.qsoff[k]),
                                    p.prow[mats[k]], p.pcol[mats[k]], dst + p.poff[mats[k]], ps));
    ++stats.kernels;
  }
  const int vecs[8] = {TPS_P_B_QKV, TPS_P_B_O, TPS_P_B_1, TPS_P_B_2, TPS_P_G1, TPS_P_BE1, TPS_P_G2, TPS_P_BE2};
  for (int k = 0; k < 8; ++k) {
    const int64_t len = p.prow[vecs[k]] * p.pcol[vecs[k]];
    if (len)
      TPS_HIP(hipMemcpyAsync(dst + p.poff[vecs[k]], q + p.qoff[vecs[k]], (size_t)len * p.esize,
                             hipMemcpyDeviceToDevice, ps));
  }
  return TPS_OK;
}

// Transposed copies of the weight matrices that an NT product reads: the
// input-gradient GEMMs whose contraction is shorter than the NN threshold
// (QKV over qw, output projection over h, up projection over uw, down
// projection over h), and with resident weights the forward down projection
// when its contraction f takes the NN form against W2^T.
int tps_stage::refresh_wt(int l, int e) {
  int ent = e;
  const char* P = params_of(l, &ent);
  char* W = wt_of(l, e);
  const int h = p.h, f = p.f, qw = (int)p.qw, uw = (int)p.uw;
  if (!nn_for(qw)) {
    TPS_HIP(transpose_launch(p.dtype, qw, h, P + p.poff[TPS_P_W_QKV], h, W + p.wtoff[0], qw, cs));
    ++stats.kernels;
  }
  if (!nn_for(h)) {
    TPS_HIP(transpose_launch(p.dtype, h, h, P + p.poff[TPS_P_W_O], h, W + p.wtoff[1], h, cs));
    ++stats.kernels;
  }
  if (!nn_for(uw)) {
    TPS_HIP(transpose_launch(p.dtype, uw, h, P + p.poff[TPS_P_W_1], h, W + p.wtoff[2], uw, cs));
    ++stats.kernels;
  }
  if (!nn_for(h) || (nn_for(f) && p.weights == TPS_W_RESIDENT)) {
    TPS_HIP(transpose_launch(p.dtype, h, f, P + p.poff[TPS_P_W_2], f, W + p.wtoff[3], h, cs));
    ++stats.kernels;
  }
  return TPS_OK;
}

// Adds (overwrite: writes) the layer's bias / LayerNorm partial sums of one
// micro-batch to its gradient block G (on the current kernel stream, the
// parameter-gradient stream in a layer backward) and clears them.
int tps_stage::finalize_bias_grads(int l, float* G, bool overwrite) {
  static const int which[Plan::BP_COUNT] = {TPS_P_B_QKV, TPS_P_B_O, TPS_P_B_1, TPS_P_B_2,
                                            TPS_P_BE1,   TPS_P_G1,  TPS_P_BE2, TPS_P_G2};
  ColMap m{};
  m.n = Plan::BP_COUNT;
  for (int r = 0; r <= Plan::BP_COUNT; ++r) m.c0[r] = (int)p.bpc[r];
  for (int r = 0; r < Plan::BP_COUNT; ++r) m.goff[r] = (int64_t)(p.goff[which[r]] / 4);
  const int k = kbegin("bias gradient finalize", 0.0, (double)p.bpart_segs * p.bpc[Plan::BP_COUNT] * 8.0);
  TPS_HIP(colsum_finalize_launch(m, bpart(l), p.bpart_segs, p.bpc[Plan::BP_COUNT], G, ks, overwrite ? 1 : 0));
  ++stats.kernels;
  return kend(k);
}

int tps_stage::flush_grads(int e) {
  WinEntry& w = win[e];
  if (w.layer < 0 || !w.grads_live) return TPS_OK;
  TPS_HIP(hipEventRecord(ev_tmp, cs));
  TPS_HIP(hipStreamWaitEvent(xs, ev_tmp, 0));
  TPS_HIP(d2h_async(lg[w.layer], grads_of(w.layer, e), p.gbytes, xs));
  stats.d2h_bytes += p.gbytes;
  TPS_HIP(hipEventRecord(w.grads_out.ev, xs));
  w.grads_out.valid = true;
  TPS_HIP(hipEventRecord(lgrads_out_ev[w.layer].ev, xs));
  lgrads_out_ev[w.layer].valid = true;
  w.grads_live = false;
  return TPS_OK;
}

int tps_stage::flush_all_grads() {
  if (p.weights != TPS_W_STREAM) return TPS_OK;
  for (size_t e = 0; e < win.size(); ++e) TPS_TRY(flush_grads((int)e));
  return TPS_OK;
}

// Make layer l's parameters resident (streamed mode); issues the H2D on the
// copy stream if needed.  Does not make the compute stream wait.
int tps_stage::prefetch_layer(int l) {
  if (p.weights != TPS_W_STREAM || l < 0 || l >= p.L) return TPS_OK;
  for (auto& w : win)
    if (w.layer == l) return TPS_OK;
  // evict the least recently used entry
  int victim = 0;
  for (size_t e = 1; e < win.size(); ++e)
    if (win[e].tick < win[victim].tick) victim = (int)e;
  WinEntry& w = win[victim];
  TPS_TRY(flush_grads(victim));
  if (w.last_use.valid) TPS_HIP(hipStreamWaitEvent(ps, w.last_use.ev, 0));
  if (p.wt_bytes) TPS_TRY(poison_fill(wt_of(l, victim), p.wt_bytes, ps));
  w.layer = l;
  w.tick = ++tick;
  w.wt_valid = false;
  TPS_TRY(wait_layer_update(l));
  TPS_TRY(load_params(l, victim));
  TPS_HIP(hipEventRecord(w.param_ready.ev, ps));
  w.param_ready.valid = true;
  w.grads_live = false;
  return TPS_OK;
}

// Marks the window entry's last compute use (cs): an eviction's H2D into
// the entry waits for it.  Every kernel sequence that reads an entry's
// parameters, transposes or gradients is followed by one.
int tps_stage::touch(int e) {
  if (e < 0) return TPS_OK;
  TPS_HIP(hipEventRecord(win[e].last_use.ev, cs));
  win[e].last_use.valid = true;
  return TPS_OK;
}

// Drops every window entry at an iteration boundary: the caller may have
// changed the host parameter blocks since the last iteration, so no layer
// may run on parameters (or transposed copies) brought in before.  The
// entries keep their last-use and grads-out events, which the next H2D and
// the next gradient fill of the entry still wait for, and their recency: the
// next iteration's first loads evict the entries the backward finished with
// first, so they overlap the end of that backward instead of waiting for it.
int tps_stage::invalidate_window() {
  for (auto& w : win) {
    w.layer = -1;
    w.wt_valid = false;
    w.grads_live = false;
    w.param_ready.valid = false;
  }
  return TPS_OK;
}

// ---------------------------------------------------------------------------
// Host optimizer (T-Offload of model state, Section 5): once every backward
// of the iteration has passed layer l, its gradient block is flushed to the
// host and a worker thread, after that copy has completed, applies one AdamW
// step to the layer's f32 master weights and moments and rewrites the pinned
// parameter block the next iteration loads (storage dtype or quantized).
// ---------------------------------------------------------------------------
int tps_stage::opt_after_backward(int l, int passes) {
  if (!hopt.on) return TPS_OK;
  hopt.bpass[l] += passes;
  if (hopt.bpass[l] < p.M) return TPS_OK;
  if (l < hopt.n_dev) {
    // on the device, in compute-stream order after the layer's last
    // backward: its gradients stay in the window entry and are consumed
    // there (not copied to the host)
    int e = 0;
    while (e < (int)win.size() && win[e].layer != l) ++e;
    if (e == (int)win.size()) return set_error(TPS_ESTATE, "device optimizer: layer not resident");
    const AdamwCoef c = adamw_coef(hopt.hp, hopt.step[l]);
    const float cf[6] = {c.b1, c.b2, c.eps, c.lr_c, c.inv_bc2_sqrt, c.wd_c};
    const float* G = grads_of(l, e);
    char* out = static_cast<char*>(hopt.dparams[l]);
    for (int i = 0; i < TPS_P_COUNT; ++i) {
      if (p.prow[i] == 0) continue;
      const int64_t n = p.prow[i] * p.pcol[i], o = (int64_t)(p.goff[i] / 4);
      TPS_HIP(adamw_launch(p.dtype, n, hopt.master[l] + o, hopt.m[l] + o, hopt.v[l] + o, G + o, out + p.poff[i], cf,
                           cs));
      ++stats.kernels;
    }
    TPS_HIP(hipEventRecord(hopt.dev_ev[l], cs));
    hopt.dev_ev_valid[l] = 1;
    ++hopt.step[l];
    win[e].grads_live = false;
    return touch(e);
  }
  for (size_t e = 0; e < win.size(); ++e)
    if (win[e].layer == l) TPS_TRY(flush_grads((int)e));
  TPS_HIP(hipEventRecord(hopt.final_ev[l], xs));
  {
    std::lock_guard<std::mutex> lock(hopt.mu);
    hopt.pending[l] = 1;
    hopt.queue.push_back(l);
  }
  hopt.cv.notify_all();
  return TPS_OK;
}

int tps_stage::wait_layer_update(int l) {
  if (!hopt.on) return TPS_OK;
  const auto t0 = std::chrono::steady_clock::now();
  std::unique_lock<std::mutex> lock(hopt.mu);
  hopt.cv.wait(lock, [&] { return !hopt.pending[l]; });
  stats.host_wait_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  if (hopt.rc != TPS_OK) return set_error(hopt.rc, "host optimizer: " + hopt.err);
  return TPS_OK;
}

int tps_stage::wait_all_updates() {
  if (!hopt.on) return TPS_OK;
  std::unique_lock<std::mutex> lock(hopt.mu);
  hopt.cv.wait(lock, [&] {
    for (char c : hopt.pending)
      if (c) return false;
    return true;
  });
  if (hopt.rc != TPS_OK) return set_error(hopt.rc, "host optimizer: " + hopt.err);
  return TPS_OK;
}

void tps_stage::opt_worker() {
  (void)hipSetDevice(device);
  for (;;) {
    int l;
    {
      std::unique_lock<std::mutex> lock(hopt.mu);
      hopt.cv.wait(lock, [&] { return hopt.stop || !hopt.queue.empty(); });
      if (hopt.queue.empty()) return;
      l = hopt.queue.front();
      hopt.queue.pop_front();
    }
    int rc = TPS_OK;
    std::string err;
    const hipError_t he = hipEventSynchronize(hopt.final_ev[l]);
    if (he != hipSuccess) {
      rc = TPS_EHIP;
      err = std::string("waiting for the gradients of layer ") + std::to_string(l) + ": " + hipGetErrorString(he);
    } else {
      const auto t0 = std::chrono::steady_clock::now();
      rc = host_adamw(p, &hopt.hp, hopt.step[l], hopt.master[l], hopt.m[l], hopt.v[l], lg[l], lp[l], p.quant,
                      hopt.threads);
      if (rc != TPS_OK) err = last_error();
      const double ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
      std::lock_guard<std::mutex> lock(hopt.mu);
      stats.host_update_ms += ms;
      ++stats.host_updates;
    }
    {
      std::lock_guard<std::mutex> lock(hopt.mu);
      ++hopt.step[l];
      hopt.pending[l] = 0;
      if (rc != TPS_OK && hopt.rc == TPS_OK) {
        hopt.rc = rc;
        hopt.err = err;
      }
    }
    hopt.cv.notify_all();
  }
}

int tps_stage::ensure_layer(int l, bool for_backward, int* entry) {
  *entry = -1;
  if (p.weights != TPS_W_STREAM) return TPS_OK;
  TPS_TRY(prefetch_layer(l));
  int e = 0;
  while (win[e].layer != l) ++e;
  WinEntry& w = win[e];
  w.tick = ++tick;
  TPS_HIP(hipStreamWaitEvent(cs, w.param_ready.ev, 0));
  if (for_backward && !w.wt_valid) {
    TPS_TRY(refresh_wt(l, e));
    w.wt_valid = true;
  }
  if (for_backward && !w.grads_live) {
    // the grad block of this entry may still be leaving for another layer
    if (w.grads_out.valid) TPS_HIP(hipStreamWaitEvent(cs, w.grads_out.ev, 0));
    if (grads_touched[l]) {
      TPS_HIP(hipEventRecord(ev_tmp, cs));
      TPS_HIP(hipStreamWaitEvent(ps, ev_tmp, 0));
      // the host block holds this layer's sums once its last flush is done
      if (lgrads_out_ev[l].valid) TPS_HIP(hipStreamWaitEvent(ps, lgrads_out_ev[l].ev, 0));
      TPS_HIP(hipMemcpyAsync(grads_of(l, e), lg[l], p.gbytes, hipMemcpyHostToDevice, ps));
      stats.h2d_bytes += p.gbytes;
      TPS_HIP(hipEventRecord(ev_tmp, ps));
      TPS_HIP(hipStreamWaitEvent(cs, ev_tmp, 0));
    } else {
      // the layer's first backward of the iteration writes every gradient
      // tensor instead of adding to it, so the block needs no zero fill
      grads_fresh[l] = 1;
      grads_touched[l] = 1;
    }
    w.grads_live = true;
  }
  *entry = e;
  return TPS_OK;
}

// ---------------------------------------------------------------------------
// Kernel timing: events recorded on the stream each selected launch goes to
// (the current kernel stream), resolved when the totals are read.
// ---------------------------------------------------------------------------
int tps_stage::kbegin(const char* name, double flops, double bytes) {
  if (!timing || strncmp(name, tprefix.c_str(), tprefix.size()) != 0) return -1;
  hipEvent_t ev[2];
  for (int i = 0; i < 2; ++i) {
    if (!tpool.empty()) {
      ev[i] = tpool.back();
      tpool.pop_back();
    } else {
      TPS_HIP(hipEventCreate(&ev[i]));
    }
  }
  TPS_HIP(hipEventRecord(ev[0], ks));
  tpending.push_back({name, flops, bytes, ev[0], ev[1], ks});
  return (int)tpending.size() - 1;
}

int tps_stage::kend(int idx) {
  if (idx < 0) return TPS_OK;
  TPS_HIP(hipEventRecord(tpending[idx].b, tpending[idx].on));
  return TPS_OK;
}

int tps_stage::kresolve() {
  for (auto& r : tpending) {
    TPS_HIP(hipEventSynchronize(r.b));
    float ms = 0.f;
    TPS_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    tps_kernel_time& a = tagg[r.name];
    if (a.launches == 0) {
      memset(&a, 0, sizeof(a));
      strncpy(a.name, r.name.c_str(), sizeof(a.name) - 1);
    }
    a.launches += 1;
    a.ms += ms;
    a.flops += r.flops;
    a.bytes += r.bytes;
    tpool.push_back(r.a);
    tpool.push_back(r.b);
  }
  tpending.clear();
  return TPS_OK;
}

// ---------------------------------------------------------------------------
// One layer forward (or a replay of part of it).
// ---------------------------------------------------------------------------
int tps_stage::fwd_layer(int l, int mb, const char* W, void* y, uint32_t ops, bool replay, bool bwd_slots) {
  const int T = p.T, h = p.h, f = p.f;
  auto ptr = [&](int t) { return tensor(l, t, mb, bwd_slots); };
  // optional outputs: in the forward written unless dropped; in a replay
  // written only when they are the tensors being regenerated
  auto opt = [&](int t) -> bool {
    const bool rec = p.pol(l, t) == TPS_RECOMPUTE;
    return replay ? rec : !rec;
  };
  const char* P = W;
  auto par = [&](int i) { return P + p.poff[i]; };
  void *x = ptr(TPS_T_X), *a = ptr(TPS_T_A), *qkv = ptr(TPS_T_QKV), *o = ptr(TPS_T_O);
  void *x1 = ptr(TPS_T_X1), *c = ptr(TPS_T_C), *u = ptr(TPS_T_U), *g = ptr(TPS_T_G);
  float* lse = static_cast<float*>(ptr(TPS_T_LSE));
  float* ln1 = static_cast<float*>(ptr(TPS_T_LN1));
  float* ln2 = static_cast<float*>(ptr(TPS_T_LN2));

  const double es = p.esize;
  const int qw = (int)p.qw, uw = (int)p.uw;
  // LLAMA layers have no biases: the residual epilogues add a zero vector
  const void* zb = p.llama ? work(p.work.zbias) : nullptr;
  auto bias = [&](int i) -> const void* { return p.llama ? zb : par(i); };
  const char* ln_name = tname("tps::ln_fwd_kernel<__bf16>", "tps::ln_fwd_kernel<float>");
  auto norm = [&](const void* in, int gi, int bi, void* out, float* st, bool keep_st) -> int {
    ++stats.kernels;
    const int k = kbegin(p.llama ? "rmsnorm forward" : ln_name, 0.0, 2.0 * T * h * es);
    if (p.llama)
      TPS_HIP(rmsnorm_fwd_launch(p.dtype, T, h, in, par(gi), p.eps, out, keep_st ? st : nullptr, ks));
    else
      TPS_HIP(layernorm_fwd_launch(p.dtype, T, h, in, par(gi), par(bi), p.eps, out, keep_st ? st : nullptr,
                                   keep_st ? st + T : nullptr, ks));
    return kend(k);
  };
  if (ops & (1u << OP_LN1)) TPS_TRY(norm(x, TPS_P_G1, TPS_P_BE1, a, ln1, opt(TPS_T_LN1)));
  if (ops & (1u << OP_QKV)) {
    if (p.llama) {
      TPS_TRY(gemm(TPS_GEMM_NT, TPS_EPI_STORE, T, qw, h, a, h, par(TPS_P_W_QKV), h, qkv, qw));
      // q and k turned in place: the stored qkv is what the attention reads
      ++stats.kernels;
      const int k = kbegin("rope", 0.0, 4.0 * T * (p.nh + p.nkv) * p.d * es);
      TPS_HIP(rope_launch(qkv, qw, T, p.s, p.nh + p.nkv, p.d, reinterpret_cast<const float*>(work(p.work.rope)), 0,
                          ks));
      TPS_TRY(kend(k));
    } else {
      TPS_TRY(gemm(TPS_GEMM_NT, TPS_EPI_BIAS, T, 3 * h, h, a, h, par(TPS_P_W_QKV), h, qkv, 3 * h, par(TPS_P_B_QKV)));
    }
  }
  if (ops & (1u << OP_ATTN)) {
    ++stats.kernels;
    const int k = kbegin(p.dtype == TPS_BF16 ? (p.d == 128 ? attention_fwd_v3_name(p.b, p.s, p.nh) : "tps::attn_fwd_v2_kernel<64>")
                                             : "tps::attn_fwd_kernel<float>",
                         2.0 * p.b * h * (double)p.s * (p.s + 1), ((double)qw + h) * T * es);
    TPS_HIP(attention_fwd_launch(p.dtype, p.b, p.s, p.nh, p.nkv, p.d, qkv, o, opt(TPS_T_LSE) ? lse : nullptr, ks));
    TPS_TRY(kend(k));
  }
  if (ops & (1u << OP_OPROJ))
    TPS_TRY(gemm(TPS_GEMM_NT, TPS_EPI_BIAS_RESID, T, h, h, o, h, par(TPS_P_W_O), h, x1, h, bias(TPS_P_B_O), x, h));
  if (ops & (1u << OP_LN2)) TPS_TRY(norm(x1, TPS_P_G2, TPS_P_BE2, c, ln2, opt(TPS_T_LN2)));
  auto swiglu = [&]() -> int {
    ++stats.kernels;
    const int k = kbegin("swiglu", 0.0, 3.0 * T * f * es);
    TPS_HIP(swiglu_launch(T, f, u, g, ks));
    return kend(k);
  };
  if (ops & (1u << OP_FC1)) {
    if (p.llama) {
      // u = [gate | up] is always materialised (the SwiGLU reads it)
      TPS_TRY(gemm(TPS_GEMM_NT, TPS_EPI_STORE, T, uw, h, c, h, par(TPS_P_W_1), h, u, uw));
      TPS_TRY(swiglu());
    } else {
      TPS_TRY(gemm(TPS_GEMM_NT, TPS_EPI_BIAS_GELU, T, f, h, c, h, par(TPS_P_W_1), h, g, f, par(TPS_P_B_1), nullptr, 0,
                   opt(TPS_T_U) ? u : nullptr, f));
    }
  }
  if (ops & (1u << OP_GELU)) {
    if (p.llama) {
      TPS_TRY(swiglu());
    } else {
      ++stats.kernels;
      const int k = kbegin(tname("tps::gelu_kernel<__bf16>", "tps::gelu_kernel<float>"), 0.0, 2.0 * T * f * es);
      TPS_HIP(gelu_launch(p.dtype, (int64_t)T * f, u, g, ks));
      TPS_TRY(kend(k));
    }
  }
  if (ops & (1u << OP_FC2)) {
    // with resident weights the transposed copies exist from the start of
    // the iteration: a long contraction reads W2^T [f][h]
    if (nn_for(f) && p.weights == TPS_W_RESIDENT)
      TPS_TRY(gemm(TPS_GEMM_NN, TPS_EPI_BIAS_RESID, T, h, f, g, f, wt_of(l, -1) + p.wtoff[3], h, y, h, bias(TPS_P_B_2),
                   x1, h));
    else
      TPS_TRY(gemm(TPS_GEMM_NT, TPS_EPI_BIAS_RESID, T, h, f, g, f, par(TPS_P_W_2), f, y, h, bias(TPS_P_B_2), x1, h));
  }
  return TPS_OK;
}

// ---------------------------------------------------------------------------
// One layer backward; parameter gradients accumulate into G (f32).
// ---------------------------------------------------------------------------
// wp: the set of intermediate-gradient buffers to use; defer: leave the
// parameter-gradient kernels running on gs at the end (they are joined before
// the buffers of set wp are written again, and once per micro-batch)
int tps_stage::bwd_layer(int l, int mb, const char* W, const char* WT, float* G, const void* dy, void* dx, int wp,
                         bool defer, int grp) {
  if (p.llama) return bwd_layer_llama(l, mb, W, WT, G, dy, dx, wp, defer, grp);
  const int T = p.T, h = p.h, f = p.f;
  ks = cs;
  const bool fresh = grads_fresh[l] != 0;
  grads_fresh[l] = 0;
  if (defer && gs_pending[wp]) {
    TPS_HIP(hipStreamWaitEvent(cs, ev_gs[wp], 0));
    gs_pending[wp] = false;
  }
  auto ptr = [&](int t) { return tensor(l, t, mb, true); };
  auto par = [&](int i) { return W + p.poff[i]; };
  auto grd = [&](int i) { return reinterpret_cast<float*>(reinterpret_cast<char*>(G) + p.goff[i]); };
  void *x = ptr(TPS_T_X), *a = ptr(TPS_T_A), *qkv = ptr(TPS_T_QKV), *o = ptr(TPS_T_O);
  void *x1 = ptr(TPS_T_X1), *c = ptr(TPS_T_C), *u = ptr(TPS_T_U), *g = ptr(TPS_T_G);
  const float* lse = static_cast<const float*>(ptr(TPS_T_LSE));
  const float* ln1 = static_cast<const float*>(ptr(TPS_T_LN1));
  const float* ln2 = static_cast<const float*>(ptr(TPS_T_LN2));
  const bool tn = grp < 0;   // weight gradients per micro-batch
  void* dx1 = tn ? work(p.work.dx1[wp]) : grp_slot(p.work.grp_dx1, p.tbytes[TPS_T_X], grp);
  void* t1 = work(p.work.t1);
  void* du = tn ? work(p.work.du[wp]) : grp_slot(p.work.grp_du, p.tbytes[TPS_T_U], grp);
  void* dqkv = tn ? work(p.work.dqkv[wp]) : grp_slot(p.work.grp_dqkv, p.tbytes[TPS_T_QKV], grp);
  float* dvec = reinterpret_cast<float*>(work(p.work.dvec));

  const double es = p.esize;
  const char* cs_name = "column sums";
  const char* lnb_name = "layernorm backward (2 kernels)";
  // bias and LayerNorm parameter gradients: per-segment column sums go to
  // the layer's partial block, summed into G by one kernel at the end
  float* bp = bpart(l);
  bpart_clean = false;
  const int64_t bstride = p.bpc[Plan::BP_COUNT];
  auto colsum = [&](const void* src, int cols, int range) -> int {
    ++stats.kernels;
    const int k = kbegin(cs_name, 0.0, (double)T * cols * es);
    TPS_HIP(colsum_acc_launch(p.dtype, T, cols, src, cols, bp + p.bpc[range], bstride, ks));
    return kend(k);
  };
  // parameter-gradient kernels on gs once what cs issued so far is done;
  // back to cs for the next input-gradient kernel
  auto to_gs = [&]() -> int {
    TPS_HIP(hipEventRecord(ev_fork, cs));
    TPS_HIP(hipStreamWaitEvent(gs, ev_fork, 0));
    ks = gs;
    return TPS_OK;
  };
  auto to_cs = [&]() { ks = cs; };
  // beta's columns precede gamma's in the partial block
  auto lnbwd = [&](const void* dout, const void* xin, const float* st, int gi, int be_range, const void* res,
                   void* dst) -> int {
    ++stats.kernels;
    const int k = kbegin(lnb_name, 0.0, 5.0 * T * h * es);
    TPS_HIP(layernorm_bwd_acc_launch(p.dtype, T, h, dout, xin, st, st + T, par(gi), res, dst, bp + p.bpc[be_range],
                                     h, bstride, cs));
    return kend(k);
  };
  // MLP: y = x1 + GeLU(c W1^T + b1) W2^T + b2
  // input gradient dX [T, N] = dY [T, K] W [K, N] for a weight W stored
  // [K][N]: an NT product against the transposed copy W^T [N][K], or for a
  // long contraction an NN product against W itself
  auto ingrad = [&](int epi, int N, int K, const void* dY, int wi, const char* wt, void* dX, void* aux) -> int {
    if (nn_for(K))
      return gemm(TPS_GEMM_NN, epi, T, N, K, dY, K, par(wi), N, dX, N, nullptr, nullptr, 0, aux, aux ? N : 0);
    return gemm(TPS_GEMM_NT, epi, T, N, K, dY, K, wt, K, dX, N, nullptr, nullptr, 0, aux, aux ? N : 0);
  };
  const char* w2t = WT + p.wtoff[3];   // [f, h]
  const char* w1t = WT + p.wtoff[2];   // [h, f]
  const char* wot = WT + p.wtoff[1];   // [h, h]
  const char* wqt = WT + p.wtoff[0];   // [h, 3h]
  // The weight and bias gradients run on gs beside the input-gradient chain
  // on cs (their inputs are only read from here on, and every buffer they
  // read is rewritten only after a join); the bias partials of gs and of the
  // LayerNorm passes on cs are disjoint columns.
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, h, f, T, dy, h, g, f, grd(TPS_P_W_2), f, nullptr, nullptr, 0, nullptr,
                 0, fresh));
  TPS_TRY(colsum(dy, h, Plan::BP_2));
  to_cs();
  TPS_TRY(ingrad(TPS_EPI_GELU_GRAD, f, h, dy, TPS_P_W_2, w2t, du, u));
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, f, h, T, du, f, c, h, grd(TPS_P_W_1), h, nullptr, nullptr, 0, nullptr,
                 0, fresh));
  TPS_TRY(colsum(du, f, Plan::BP_1));
  to_cs();
  TPS_TRY(ingrad(TPS_EPI_STORE, h, f, du, TPS_P_W_1, w1t, t1, nullptr));
  TPS_TRY(lnbwd(t1, x1, ln2, TPS_P_G2, Plan::BP_BE2, dy, dx1));
  // attention block: x1 = x + o Wo^T + bo
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, h, h, T, dx1, h, o, h, grd(TPS_P_W_O), h, nullptr, nullptr, 0, nullptr,
                 0, fresh));
  TPS_TRY(colsum(dx1, h, Plan::BP_O));
  to_cs();
  TPS_TRY(ingrad(TPS_EPI_STORE, h, h, dx1, TPS_P_W_O, wot, t1, nullptr));
  {
    ++stats.kernels;
    const int k = kbegin("attention backward", 4.0 * p.b * h * (double)p.s * (p.s + 1), 9.0 * T * h * es);
    TPS_HIP(attention_bwd_launch(p.dtype, p.b, p.s, p.nh, p.nh, p.d, qkv, o, lse, t1, dqkv, dvec, nullptr, cs));
    TPS_TRY(kend(k));
  }
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, 3 * h, h, T, dqkv, 3 * h, a, h, grd(TPS_P_W_QKV), h, nullptr, nullptr,
                 0, nullptr, 0, fresh));
  TPS_TRY(colsum(dqkv, 3 * h, Plan::BP_QKV));
  to_cs();
  TPS_TRY(ingrad(TPS_EPI_STORE, h, 3 * h, dqkv, TPS_P_W_QKV, wqt, t1, nullptr));
  TPS_TRY(lnbwd(t1, x, ln1, TPS_P_G1, Plan::BP_BE1, dx1, dx));
  // finalize after both streams' column sums; cs continues at once (defer)
  // or once gs is done
  TPS_TRY(to_gs());
  TPS_TRY(finalize_bias_grads(l, G, fresh));
  to_cs();
  if (defer) {
    TPS_HIP(hipEventRecord(ev_gs[wp], gs));
    gs_pending[wp] = true;
    gs_layer[wp] = l;
  } else {
    TPS_TRY(join_gs());
  }
  bpart_clean = true;
  return TPS_OK;
}

// LLAMA-style layer backward: the same stream protocol as bwd_layer (weight
// gradients forked to gs as their inputs appear, lazily joined), with the
// SwiGLU and rotary backward kernels in the input-gradient chain and only the
// two RMSNorm gains among the vector parameters.
int tps_stage::bwd_layer_llama(int l, int mb, const char* W, const char* WT, float* G, const void* dy, void* dx,
                               int wp, bool defer, int grp) {
  const int T = p.T, h = p.h, f = p.f, qw = (int)p.qw, uw = (int)p.uw;
  ks = cs;
  const bool fresh = grads_fresh[l] != 0;
  grads_fresh[l] = 0;
  if (defer && gs_pending[wp]) {
    TPS_HIP(hipStreamWaitEvent(cs, ev_gs[wp], 0));
    gs_pending[wp] = false;
  }
  auto ptr = [&](int t) { return tensor(l, t, mb, true); };
  auto par = [&](int i) { return W + p.poff[i]; };
  auto grd = [&](int i) { return reinterpret_cast<float*>(reinterpret_cast<char*>(G) + p.goff[i]); };
  void *x = ptr(TPS_T_X), *a = ptr(TPS_T_A), *qkv = ptr(TPS_T_QKV), *o = ptr(TPS_T_O);
  void *x1 = ptr(TPS_T_X1), *c = ptr(TPS_T_C), *u = ptr(TPS_T_U), *g = ptr(TPS_T_G);
  const float* lse = static_cast<const float*>(ptr(TPS_T_LSE));
  const float* r1 = static_cast<const float*>(ptr(TPS_T_LN1));
  const float* r2 = static_cast<const float*>(ptr(TPS_T_LN2));
  const bool tn = grp < 0;   // weight gradients per micro-batch
  void* dx1 = tn ? work(p.work.dx1[wp]) : grp_slot(p.work.grp_dx1, p.tbytes[TPS_T_X], grp);
  void* t1 = work(p.work.t1);
  void* du = tn ? work(p.work.du[wp]) : grp_slot(p.work.grp_du, p.tbytes[TPS_T_U], grp);
  void* dqkv = tn ? work(p.work.dqkv[wp]) : grp_slot(p.work.grp_dqkv, p.tbytes[TPS_T_QKV], grp);
  void* dg = work(p.work.dg);
  void* kvws = p.work.kvws == kNone ? nullptr : work(p.work.kvws);
  const float* rope_tab = reinterpret_cast<const float*>(work(p.work.rope));
  float* dvec = reinterpret_cast<float*>(work(p.work.dvec));
  const double es = p.esize;
  float* bp = bpart(l);
  bpart_clean = false;
  const int64_t bstride = p.bpc[Plan::BP_COUNT];
  auto to_gs = [&]() -> int {
    TPS_HIP(hipEventRecord(ev_fork, cs));
    TPS_HIP(hipStreamWaitEvent(gs, ev_fork, 0));
    ks = gs;
    return TPS_OK;
  };
  auto to_cs = [&]() { ks = cs; };
  // dst = res + RMSNorm^T(dout); the gain's per-segment sums go to its
  // columns of the layer's partial block
  auto rmsbwd = [&](const void* dout, const void* xin, const float* rstd, int gi, int range, const void* res,
                    void* dst) -> int {
    ++stats.kernels;
    const int k = kbegin("rmsnorm backward (2 kernels)", 0.0, 5.0 * T * h * es);
    TPS_HIP(rmsnorm_bwd_acc_launch(p.dtype, T, h, dout, xin, rstd, par(gi), res, dst, bp + p.bpc[range], bstride,
                                   cs));
    return kend(k);
  };
  auto ingrad = [&](int N, int K, const void* dY, int wi, const char* wt, void* dX) -> int {
    if (nn_for(K)) return gemm(TPS_GEMM_NN, TPS_EPI_STORE, T, N, K, dY, K, par(wi), N, dX, N);
    return gemm(TPS_GEMM_NT, TPS_EPI_STORE, T, N, K, dY, K, wt, K, dX, N);
  };
  const char* w2t = WT + p.wtoff[3];   // [f, h]
  const char* w1t = WT + p.wtoff[2];   // [h, 2f]
  const char* wot = WT + p.wtoff[1];   // [h, h]
  const char* wqt = WT + p.wtoff[0];   // [h, qw]
  // MLP: y = x1 + (SiLU(gate) * up) W2^T, [gate | up] = c W1^T
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, h, f, T, dy, h, g, f, grd(TPS_P_W_2), f, nullptr, nullptr, 0, nullptr,
                 0, fresh));
  to_cs();
  TPS_TRY(ingrad(f, h, dy, TPS_P_W_2, w2t, dg));
  {
    ++stats.kernels;
    const int k = kbegin("swiglu backward", 0.0, 5.0 * T * f * es);
    TPS_HIP(swiglu_bwd_launch(T, f, dg, u, du, cs));
    TPS_TRY(kend(k));
  }
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, uw, h, T, du, uw, c, h, grd(TPS_P_W_1), h, nullptr, nullptr, 0, nullptr,
                 0, fresh));
  to_cs();
  TPS_TRY(ingrad(h, uw, du, TPS_P_W_1, w1t, t1));
  TPS_TRY(rmsbwd(t1, x1, r2, TPS_P_G2, Plan::BP_G2, dy, dx1));
  // attention block: x1 = x + o Wo^T
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, h, h, T, dx1, h, o, h, grd(TPS_P_W_O), h, nullptr, nullptr, 0, nullptr,
                 0, fresh));
  to_cs();
  TPS_TRY(ingrad(h, h, dx1, TPS_P_W_O, wot, t1));
  {
    ++stats.kernels;
    const int k = kbegin("attention backward", 4.0 * p.b * h * (double)p.s * (p.s + 1), (3.0 * qw + 4.0 * h) * T * es);
    TPS_HIP(attention_bwd_launch(p.dtype, p.b, p.s, p.nh, p.nkv, p.d, qkv, o, lse, t1, dqkv, dvec, kvws, cs));
    TPS_TRY(kend(k));
  }
  {
    // gradients of the rotated q and k turned back to those of the projections
    ++stats.kernels;
    const int k = kbegin("rope", 0.0, 4.0 * T * (p.nh + p.nkv) * p.d * es);
    TPS_HIP(rope_launch(dqkv, qw, T, p.s, p.nh + p.nkv, p.d, rope_tab, 1, cs));
    TPS_TRY(kend(k));
  }
  TPS_TRY(to_gs());
  if (tn)
    TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, qw, h, T, dqkv, qw, a, h, grd(TPS_P_W_QKV), h, nullptr, nullptr, 0,
                 nullptr, 0, fresh));
  to_cs();
  TPS_TRY(ingrad(h, qw, dqkv, TPS_P_W_QKV, wqt, t1));
  TPS_TRY(rmsbwd(t1, x, r1, TPS_P_G1, Plan::BP_G1, dx1, dx));
  TPS_TRY(to_gs());
  TPS_TRY(finalize_bias_grads(l, G, fresh));
  to_cs();
  if (defer) {
    TPS_HIP(hipEventRecord(ev_gs[wp], gs));
    gs_pending[wp] = true;
    gs_layer[wp] = l;
  } else {
    TPS_TRY(join_gs());
  }
  bpart_clean = true;
  return TPS_OK;
}

// The four weight-gradient products of layer l over the n micro-batches of a
// backward group (K = n T): the slots of each operand are consecutive, so
// micro-batch i's rows follow micro-batch i - 1's; fresh: the first
// contribution of the iteration (writes instead of adding).
int tps_stage::batched_wgrad(int l, float* G, int n, bool fresh, int yin) {
  const int h = p.h, f = p.f, qw = (int)p.qw, uw = (int)p.uw;
  const int K = n * p.T;
  auto grd = [&](int i) { return reinterpret_cast<float*>(reinterpret_cast<char*>(G) + p.goff[i]); };
  auto base = [&](uint64_t off) { return static_cast<const void*>(arena + p.off_work + off); };
  (void)l;
  ks = cs;
  TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, h, f, K, base(p.work.grp_y[yin]), h, base(p.work.grp_act[3]), f,
               grd(TPS_P_W_2), f, nullptr, nullptr, 0, nullptr, 0, fresh));
  TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, uw, h, K, base(p.work.grp_du), uw, base(p.work.grp_act[2]), h,
               grd(TPS_P_W_1), h, nullptr, nullptr, 0, nullptr, 0, fresh));
  TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, h, h, K, base(p.work.grp_dx1), h, base(p.work.grp_act[1]), h,
               grd(TPS_P_W_O), h, nullptr, nullptr, 0, nullptr, 0, fresh));
  TPS_TRY(gemm(TPS_GEMM_TN, TPS_EPI_ACC_F32, qw, h, K, base(p.work.grp_dqkv), qw, base(p.work.grp_act[0]), h,
               grd(TPS_P_W_QKV), h, nullptr, nullptr, 0, nullptr, 0, fresh));
  return TPS_OK;
}

// ---------------------------------------------------------------------------
// Offload engine
// ---------------------------------------------------------------------------
int tps_stage::d2h_layer(int l, int mb) {
  bool any = false;
  for (int t = 0; t < TPS_T_COUNT; ++t) any |= p.oslot_off[(size_t)l * TPS_T_COUNT + t] != kNone;
  if (!any) return TPS_OK;
  TPS_HIP(hipEventRecord(ev_tmp, cs));
  TPS_HIP(hipStreamWaitEvent(xs, ev_tmp, 0));
  // the host slot may still be read by the prefetch of its previous micro-batch
  const SlotEvent& hs = hslot_read_ev[p.host_slot[mb]];
  if (hs.valid) TPS_HIP(hipStreamWaitEvent(xs, hs.ev, 0));
  for (int t = 0; t < TPS_T_COUNT; ++t) {
    const size_t k = (size_t)l * TPS_T_COUNT + t;
    if (p.oslot_off[k] == kNone) continue;
    TPS_HIP(d2h_async(host_base(mb) + p.oslot_off[k], oslot_base(p.oslot_f[mb]) + p.oslot_off[k], p.tbytes[t], xs));
    stats.d2h_bytes += p.tbytes[t];
  }
  TPS_HIP(hipEventRecord(offloaded_ev[mb].ev, xs));
  offloaded_ev[mb].valid = true;
  return TPS_OK;
}

// Bring an offloaded micro-batch back into its staging slot, deepest layer
// first (the backward starts there); one ready event per layer.
int tps_stage::prefetch_mb(int mb) {
  if (prefetched[mb]) return TPS_OK;
  const int slot = p.oslot_b[mb];
  TPS_TRY(acquire_oslot(slot, ps));
  // the micro-batch's own offload must have reached the host
  if (offloaded_ev[mb].valid) TPS_HIP(hipStreamWaitEvent(ps, offloaded_ev[mb].ev, 0));
  for (int l = p.L - 1; l >= 0; --l) {
    for (int t = 0; t < TPS_T_COUNT; ++t) {
      const size_t k = (size_t)l * TPS_T_COUNT + t;
      if (p.oslot_off[k] == kNone) continue;
      TPS_HIP(hipMemcpyAsync(oslot_base(slot) + p.oslot_off[k], host_base(mb) + p.oslot_off[k], p.tbytes[t],
                             hipMemcpyHostToDevice, ps));
      stats.h2d_bytes += p.tbytes[t];
    }
    TPS_HIP(hipEventRecord(ready_ev[mb][l], ps));
  }
  TPS_HIP(hipEventRecord(hslot_read_ev[p.host_slot[mb]].ev, ps));
  hslot_read_ev[p.host_slot[mb]].valid = true;
  prefetched[mb] = 1;
  return TPS_OK;
}

int tps_stage::run_prefetches(int pos) {
  for (int mb : p.prefetch_at[pos]) TPS_TRY(prefetch_mb(mb));
  return TPS_OK;
}

int tps_stage::check_op(int kind, int mb) {
  if (!in_iteration) return set_error(TPS_ESTATE, "call tps_stage_begin_iteration first");
  if (mb < 0 || mb >= p.M) return set_error(TPS_EORDER, "micro-batch index out of range");
  const char* name = kind == TPS_OP_F ? "F" : "B";
  if (kind == TPS_OP_B && !f_done[mb]) return set_error(TPS_EORDER, "backward before forward of micro-batch " + std::to_string(mb));
  if (kind == TPS_OP_B && b_done[mb]) return set_error(TPS_EORDER, "second backward of micro-batch " + std::to_string(mb));
  if (kind == TPS_OP_F && f_done[mb]) return set_error(TPS_EORDER, "second forward of micro-batch " + std::to_string(mb) + " in one iteration");
  if (cursor >= (int)p.op_kind.size() || p.op_kind[cursor] != kind || p.op_mb[cursor] != mb) {
    std::string want = cursor < (int)p.op_kind.size()
                           ? std::string(p.op_kind[cursor] == TPS_OP_F ? "F(" : "B(") + std::to_string(p.op_mb[cursor]) + ")"
                           : "end of iteration";
    return set_error(TPS_EORDER, std::string("call ") + name + "(" + std::to_string(mb) + ") out of the planned order; expected " + want);
  }
  return TPS_OK;
}

// ---------------------------------------------------------------------------
// F(mb) and B(mb)
// ---------------------------------------------------------------------------
int tps_stage::forward_one(int mb, const void* x, void* y) {
  const bool off = p.host_slot[mb] >= 0;
  // a forward may reuse the saved-tensor slot of a micro-batch whose last
  // parameter-gradient kernels are still running
  TPS_TRY(join_if_pending());
  if (p.oslot_bytes) TPS_TRY(acquire_oslot(p.oslot_f[mb], cs));
  TPS_HIP(hipMemcpyAsync(tensor(0, TPS_T_X, mb, false), x, p.tbytes[TPS_T_X], hipMemcpyDeviceToDevice, cs));
  for (int l = 0; l < p.L; ++l) {
    int e = -1;
    TPS_TRY(ensure_layer(l, false, &e));
    TPS_TRY(prefetch_layer(l + 1));
    void* yl = (l == p.L - 1) ? y : tensor(l + 1, TPS_T_X, mb, false);
    TPS_TRY(fwd_layer(l, mb, params_of(l, &e), yl, 0xFFu & ~(1u << OP_GELU), false, false));
    TPS_TRY(touch(e));
    if (off) TPS_TRY(d2h_layer(l, mb));
  }
  if (off) TPS_TRY(release_oslot(p.oslot_f[mb], xs));
  return TPS_OK;
}

int tps_stage::backward_one(int mb, const void* dy, void* dx) {
  const bool off = p.host_slot[mb] >= 0;
  if (off) {
    TPS_TRY(prefetch_mb(mb));
    for (int l = 0; l < p.L; ++l) TPS_HIP(hipStreamWaitEvent(cs, ready_ev[mb][l], 0));
  }
  const bool defer = p.defer_join;
  bool rs_forked = false;
  // Replay of layer l (segment granularity).  With deferred joins the
  // previous micro-batch's last layer backwards may still read its replayed
  // tensors: wait for their kernels first.  side: on rs, starting where cs is
  // now (this micro-batch's inputs and prefetched tensors in place), waited
  // for by cs before the layer's backward.
  auto replay = [&](int l, bool side) -> int {
    if (side) {
      if (!rs_forked) {
        TPS_HIP(hipEventRecord(ev_rfork, cs));
        TPS_HIP(hipStreamWaitEvent(rs, ev_rfork, 0));
        rs_forked = true;
      }
      TPS_TRY(wait_gs_layer_on(l, rs));
      ks = rs;
    } else if (defer) {
      TPS_TRY(wait_gs_layer(l));
    }
    int e = -1;
    TPS_TRY(ensure_layer(l, false, &e));
    void* yl = (l == p.L - 1) ? nullptr : tensor(l + 1, TPS_T_X, mb, true);
    TPS_TRY(fwd_layer(l, mb, params_of(l, &e), yl, p.replay_ops[l], true, true));
    if (side) {
      TPS_HIP(hipEventRecord(ev_replay[l], rs));
      replay_on_rs[l] = 1;
      ks = cs;
    }
    ++stats.replays;
    TPS_TRY(touch(e));
    return TPS_OK;
  };
  if (p.granularity == TPS_GRAN_SEGMENT) {
    if (rs) {
      // the top replayed layer on cs, the lower ones on rs beside the
      // backward of the layers above them
      bool top = true;
      for (int l = p.L - 1; l >= 0; --l) {
        if (!p.replay_ops[l]) continue;
        TPS_TRY(replay(l, !top));
        top = false;
      }
    } else {
      // top-down where the layers are independent, so the layers whose
      // lagging kernels were issued last are replayed last
      const bool down = defer && p.replay_independent;
      for (int i = 0; i < p.L; ++i) {
        const int l = down ? p.L - 1 - i : i;
        if (p.replay_ops[l]) TPS_TRY(replay(l, false));
      }
    }
  }
  // running input gradient: with deferred joins three buffers rotate over the
  // iteration's layer backwards, so the one a layer backward writes was last
  // read two layer backwards earlier (by kernels the wait at the start of
  // bwd_layer has joined), else two alternate
  const void* cur = dy;
  char* gb[3] = {work(p.work.g[0]), work(p.work.g[1]), work(p.work.g[2])};
  for (int l = p.L - 1; l >= 0; --l) {
    int e = -1;
    TPS_TRY(ensure_layer(l, true, &e));
    TPS_TRY(prefetch_layer(l - 1));
    const char* W = params_of(l, &e);
    if (p.granularity == TPS_GRAN_LAYER && p.replay_ops[l]) {
      TPS_TRY(fwd_layer(l, mb, W, nullptr, p.replay_ops[l], true, true));
      ++stats.replays;
    }
    if (rs && replay_on_rs[l]) {
      TPS_HIP(hipStreamWaitEvent(cs, ev_replay[l], 0));
      replay_on_rs[l] = 0;
    }
    void* out = (l == 0) ? dx : defer ? gb[bstep % 3] : (cur == gb[0] ? gb[1] : gb[0]);
    TPS_TRY(bwd_layer(l, mb, W, wt_of(l, e), grads_of(l, e), cur, out, defer ? (bstep & 1) : 0, defer));
    ++bstep;
    TPS_TRY(touch(e));
    TPS_TRY(opt_after_backward(l, 1));
    cur = out;
  }
  // Pending now: the parameter-gradient kernels of the last two layer
  // backwards (bottom layers), which read this micro-batch's saved tensors
  // and, with fewer than three layers, the caller's dy.  Its staging slot is
  // handed back on gs, after them; later forwards, the next replay of those
  // layers and the end of the iteration wait for them.
  if (defer && p.L < 3) TPS_TRY(join_gs());
  if (p.oslot_bytes) TPS_TRY(release_oslot(p.oslot_b[mb], defer ? gs : cs));
  return poison_after_backward(mb);
}

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" int tps_stage_init(const tps_config* cfg, const tps_params* params, const tps_memory* mem,
                              tps_stage** out) {
  clear_error();
  if (!out || !params || !mem) return set_error(TPS_EINVAL, "tps_stage_init: null argument");
  *out = nullptr;
  tps_stage* st = new (std::nothrow) tps_stage();
  if (!st) return set_error(TPS_ENOMEM, "tps_stage_init: host allocation");
  int rc = make_plan(cfg, &st->p);
  if (rc) { delete st; return rc; }
  const Plan& p = st->p;
  {
    const char* ev = std::getenv("TPS_POISON");
    st->poison = ev && *ev && std::strcmp(ev, "0") != 0;
  }
  if (!params->layer_params || !params->layer_grads) { delete st; return set_error(TPS_EINVAL, "tps_stage_init: params"); }
  for (int l = 0; l < p.L; ++l) {
    if (!params->layer_params[l] || !params->layer_grads[l]) { delete st; return set_error(TPS_EINVAL, "tps_stage_init: null layer block"); }
    st->lp.push_back(static_cast<char*>(params->layer_params[l]));
    st->lg.push_back(params->layer_grads[l]);
  }
  if (!mem->device_arena || mem->device_bytes < p.arena_bytes) {
    delete st;
    return set_error(TPS_ENOMEM, "tps_stage_init: device arena of " + std::to_string(mem->device_bytes) +
                                     " bytes, plan needs " + std::to_string(p.arena_bytes));
  }
  if ((reinterpret_cast<uintptr_t>(mem->device_arena) & 255u) != 0) { delete st; return set_error(TPS_EINVAL, "device arena must be 256-byte aligned"); }
  if (p.host_bytes && (!mem->host_arena || mem->host_bytes < p.host_bytes)) {
    delete st;
    return set_error(TPS_ENOMEM, "tps_stage_init: pinned host arena of " + std::to_string(mem->host_bytes) +
                                     " bytes, plan needs " + std::to_string(p.host_bytes));
  }
  st->arena = static_cast<char*>(mem->device_arena);
  st->host = static_cast<char*>(mem->host_arena);
  st->cs = static_cast<hipStream_t>(mem->compute_stream);
  const bool link = p.host_bytes || p.weights == TPS_W_STREAM;
  if (link && ((mem->copy_stream && mem->copy_stream == mem->compute_stream) ||
               (mem->prefetch_stream && mem->prefetch_stream == mem->compute_stream))) {
    delete st;
    return set_error(TPS_EINVAL, "offload and streamed weights need copy streams distinct from the compute stream");
  }
  auto mkev = [&](hipEvent_t* e) { return hipEventCreateWithFlags(e, hipEventDisableTiming); };
  hipError_t he = hipGetDevice(&st->device);
  if (he == hipSuccess) he = mkev(&st->ev_tmp);
  // fork and join events order kernels of two streams on this device: no
  // system-scope fence (kernel completion already releases at device scope)
  auto mkev_dev = [&](hipEvent_t* e) {
    return hipEventCreateWithFlags(e, hipEventDisableTiming | hipEventDisableSystemFence);
  };
  if (he == hipSuccess) he = mkev_dev(&st->ev_fork);
  if (he == hipSuccess) he = mkev_dev(&st->ev_join);
  for (auto& e : st->ev_gs)
    if (he == hipSuccess) he = mkev_dev(&e);
  // a replay stream when replays are light (no GEMM in any layer's replay
  // program) and independent across layers: full-layer replays beside the
  // backward slowed it down (they compete for the CUs with its critical path)
  bool light = true;
  for (int l = 0; l < p.L; ++l)
    light = light && !(p.replay_ops[l] & ((1u << OP_QKV) | (1u << OP_OPROJ) | (1u << OP_FC1) | (1u << OP_FC2)));
  if (p.defer_join && p.granularity == TPS_GRAN_SEGMENT && p.replay_independent && p.n_replay_layers > 1 && light) {
    if (he == hipSuccess) he = queue_stream(st->device, &st->rs);
    if (he == hipSuccess) he = mkev_dev(&st->ev_rfork);
    st->ev_replay.assign(p.L, nullptr);
    st->replay_on_rs.assign(p.L, 0);
    for (auto& e : st->ev_replay)
      if (he == hipSuccess) he = mkev_dev(&e);
  }
  // parameter-gradient kernels: a stream of their own, or the compute stream
  if (p.wgrad_inline) st->gs = st->cs;
  else if (he == hipSuccess) he = queue_stream(st->device, &st->gs);
  if (link) {
    st->xs = static_cast<hipStream_t>(mem->copy_stream);
    st->ps = static_cast<hipStream_t>(mem->prefetch_stream);
    if (he == hipSuccess && !st->xs && (he = queue_stream(st->device, &st->xs)) == hipSuccess) st->own_xs = true;
    if (he == hipSuccess && !st->ps && (he = queue_stream(st->device, &st->ps)) == hipSuccess) st->own_ps = true;
  }
  st->ks = st->cs;
  st->oslot_ev.resize(p.n_oslots);
  st->offloaded_ev.resize(p.M);
  st->hslot_read_ev.resize(p.n_host_slots);
  st->lgrads_out_ev.resize(p.L);
  for (auto* v : {&st->oslot_ev, &st->offloaded_ev, &st->hslot_read_ev, &st->lgrads_out_ev})
    for (auto& s : *v)
      if (he == hipSuccess) he = mkev(&s.ev);
  st->ready_ev.assign(p.M, std::vector<hipEvent_t>(p.L, nullptr));
  for (int mb = 0; mb < p.M && he == hipSuccess; ++mb)
    if (p.host_slot[mb] >= 0)
      for (int l = 0; l < p.L && he == hipSuccess; ++l) he = mkev(&st->ready_ev[mb][l]);
  if (p.weights == TPS_W_STREAM) {
    st->win.resize(p.window);
    for (auto& w : st->win) {
      if (he == hipSuccess) he = mkev(&w.param_ready.ev);
      if (he == hipSuccess) he = mkev(&w.last_use.ev);
      if (he == hipSuccess) he = mkev(&w.grads_out.ev);
    }
  }
  if (he != hipSuccess) {
    int r = check_hip(he, "tps_stage_init: stream and event creation");
    tps_stage_destroy(st);
    return r;
  }
  st->f_done.assign(p.M, 0);
  st->b_done.assign(p.M, 0);
  st->prefetched.assign(p.M, 0);
  st->grads_touched.assign(p.L, 0);
  st->grads_fresh.assign(p.L, 0);
  *out = st;
  return TPS_OK;
}

extern "C" int tps_stage_begin_iteration(tps_stage* st, int zero_grads) {
  clear_error();
  if (!st) return set_error(TPS_EINVAL, "null stage");
  if (st->hopt.on && st->hopt.n_dev > 0 && !zero_grads)
    return set_error(TPS_EINVAL, "tps_stage_begin_iteration: layers updated on the device need zero_grads");
  if (st->in_iteration && st->cursor != 0 && st->cursor < (int)st->p.op_kind.size())
    return set_error(TPS_ESTATE, "previous iteration has unfinished ops");
  st->cursor = 0;
  std::fill(st->f_done.begin(), st->f_done.end(), 0);
  std::fill(st->b_done.begin(), st->b_done.end(), 0);
  std::fill(st->prefetched.begin(), st->prefetched.end(), 0);
  {
    std::lock_guard<std::mutex> lock(st->hopt.mu);
    st->stats = tps_stats{};
  }
  const Plan& p = st->p;
  std::fill(st->hopt.bpass.begin(), st->hopt.bpass.end(), 0);
  // an iteration cut short may leave parameter-gradient kernels pending
  TPS_TRY(st->join_if_pending());
  st->bstep = 0;
  if (!st->bpart_clean) {
    // first iteration, or a layer backward was cut short by an error
    hipError_t e = fill_zero_launch(st->arena + p.off_bpart, (uint64_t)p.L * p.bpart_bytes, st->cs);
    if (e != hipSuccess) return check_hip(e, "clear bias partials");
    ++st->stats.kernels;
    st->bpart_clean = true;
  }
  if (p.llama && !st->llama_tables) {
    // the rotation table and the zero vector of the bias-free residual
    // epilogues, once per stage
    hipError_t e = rope_table_launch(p.s, p.d, p.rope_base, reinterpret_cast<float*>(st->work(p.work.rope)), st->cs);
    if (e == hipSuccess) e = fill_zero_launch(st->work(p.work.zbias), (uint64_t)p.h * p.esize, st->cs);
    if (e != hipSuccess) return check_hip(e, "rotation table");
    st->stats.kernels += 2;
    st->llama_tables = true;
  }
  if (p.weights == TPS_W_STREAM) {
    // host gradients of the previous iteration must be complete before reuse
    int rc = st->flush_all_grads();
    if (rc) return rc;
    // parameters may have changed since the last iteration: every layer is
    // brought in again (and its transposed copies rebuilt)
    rc = st->invalidate_window();
    if (rc) return rc;
    std::fill(st->grads_touched.begin(), st->grads_touched.end(), zero_grads ? 0 : 1);
  } else {
    // the first layer backward of the iteration writes each gradient tensor
    if (zero_grads) std::fill(st->grads_fresh.begin(), st->grads_fresh.end(), 1);
    // parameters may have changed since the last iteration
    for (int l = 0; l < p.L; ++l) {
      int rc = st->refresh_wt(l, -1);
      if (rc) return rc;
    }
  }
  st->in_iteration = true;
  return TPS_OK;
}

static int finish_op(tps_stage* st) {
  ++st->cursor;
  st->stats.ops_done = st->cursor;
  if (st->cursor == (int)st->p.op_kind.size()) {
    // gradients complete in compute-stream order at the end of the iteration
    TPS_TRY(st->join_if_pending());
    return st->flush_all_grads();
  }
  return TPS_OK;
}

extern "C" int tps_stage_forward(tps_stage* st, int mb, const void* x, void* y) {
  clear_error();
  if (!st) return set_error(TPS_EINVAL, "null stage");
  if (!x || !y) return set_error(TPS_EINVAL, "tps_stage_forward: null x or y");
  TPS_TRY(st->check_op(TPS_OP_F, mb));
  TPS_TRY(st->run_prefetches(st->cursor));
  TPS_TRY(st->forward_one(mb, x, y));
  st->f_done[mb] = 1;
  return finish_op(st);
}

extern "C" int tps_stage_backward(tps_stage* st, int mb, const void* dy, void* dx) {
  clear_error();
  if (!st) return set_error(TPS_EINVAL, "null stage");
  if (!dy || !dx) return set_error(TPS_EINVAL, "tps_stage_backward: null dy or dx");
  TPS_TRY(st->check_op(TPS_OP_B, mb));
  TPS_TRY(st->run_prefetches(st->cursor));
  TPS_TRY(st->backward_one(mb, dy, dx));
  st->b_done[mb] = 1;
  return finish_op(st);
}

// Layer-major groups: all micro-batches of the group go through layer l
// before layer l+1 (resp. l-1), so a streamed layer is brought in once.
extern "C" int tps_stage_forward_group(tps_stage* st, int mb0, int n, const void* const* x, void* const* y) {
  clear_error();
  if (!st || !x || !y || n < 1) return set_error(TPS_EINVAL, "tps_stage_forward_group: arguments");
  const Plan& p = st->p;
  // validate the whole group against the order first
  for (int i = 0; i < n; ++i) {
    const int pos = st->cursor + i;
    if (pos >= (int)p.op_kind.size() || p.op_kind[pos] != TPS_OP_F || p.op_mb[pos] != mb0 + i)
      return set_error(TPS_EORDER, "forward group does not match the planned order");
    if (!x[i] || !y[i]) return set_error(TPS_EINVAL, "forward group: null buffer");
  }
  TPS_TRY(st->check_op(TPS_OP_F, mb0));
  // a preceding per-micro-batch backward may have left parameter-gradient
  // kernels running that still read slots and buffers this group rewrites
  TPS_TRY(st->join_if_pending());
  if (n > 1)
    for (int l = 1; l < p.L; ++l)
      if (p.pol(l, TPS_T_X) == TPS_RECOMPUTE)
        return set_error(TPS_EINVAL, "forward groups of more than one micro-batch need every layer input kept or offloaded");
  for (int i = 0; i < n; ++i) TPS_TRY(st->run_prefetches(st->cursor + i));
  for (int i = 0; i < n; ++i) {
    const int mb = mb0 + i;
    if (p.oslot_bytes) TPS_TRY(st->acquire_oslot(p.oslot_f[mb], st->cs));
    TPS_HIP(hipMemcpyAsync(st->tensor(0, TPS_T_X, mb, false), x[i], p.tbytes[TPS_T_X], hipMemcpyDeviceToDevice, st->cs));
  }
  for (int l = 0; l < p.L; ++l) {
    int e = -1;
    TPS_TRY(st->ensure_layer(l, false, &e));
    TPS_TRY(st->prefetch_layer(l + 1));
    for (int i = 0; i < n; ++i) {
      const int mb = mb0 + i;
      void* yl = (l == p.L - 1) ? y[i] : st->tensor(l + 1, TPS_T_X, mb, false);
      TPS_TRY(st->fwd_layer(l, mb, st->params_of(l, &e), yl, 0xFFu & ~(1u << OP_GELU), false, false));
      if (p.host_slot[mb] >= 0) TPS_TRY(st->d2h_layer(l, mb));
    }
    TPS_TRY(st->touch(e));
  }
  for (int i = 0; i < n; ++i) {
    const int mb = mb0 + i;
    if (p.host_slot[mb] >= 0) TPS_TRY(st->release_oslot(p.oslot_f[mb], st->xs));
    st->f_done[mb] = 1;
    ++st->cursor;
  }
  st->stats.ops_done = st->cursor;
  if (st->cursor == (int)p.op_kind.size()) return st->flush_all_grads();
  return TPS_OK;
}

extern "C" int tps_stage_backward_group(tps_stage* st, int mb0, int n, const void* const* dy, void* const* dx) {
  clear_error();
  if (!st || !dy || !dx || n < 1) return set_error(TPS_EINVAL, "tps_stage_backward_group: arguments");
  const Plan& p = st->p;
  for (int i = 0; i < n; ++i) {
    const int pos = st->cursor + i;
    if (pos >= (int)p.op_kind.size() || p.op_kind[pos] != TPS_OP_B || p.op_mb[pos] != mb0 + i)
      return set_error(TPS_EORDER, "backward group does not match the planned order");
    if (!st->f_done[mb0 + i]) return set_error(TPS_EORDER, "backward before forward in group");
    if (!dy[i] || !dx[i]) return set_error(TPS_EINVAL, "backward group: null buffer");
  }
  TPS_TRY(st->check_op(TPS_OP_B, mb0));
  if (p.granularity == TPS_GRAN_SEGMENT && n > 1) {
    bool any = false;
    for (int l = 0; l < p.L; ++l) any |= p.replay_ops[l] != 0;
    if (any) return set_error(TPS_EINVAL, "segment replay shares one replay buffer: backward groups of more than one micro-batch need layer granularity");
  }
  // the layer backwards below write work set 0 and the running-gradient
  // buffer, which lagging parameter-gradient kernels of a preceding
  // per-micro-batch backward may still read
  TPS_TRY(st->join_if_pending());
  for (int i = 0; i < n; ++i) TPS_TRY(st->run_prefetches(st->cursor + i));
  // gradients flow per micro-batch through ping-pong buffers; keep one pair
  // per group member in the caller's dx buffers: dx[i] holds the running
  // gradient of micro-batch i between layers.
  for (int i = 0; i < n; ++i) {
    const int mb = mb0 + i;
    if (p.host_slot[mb] >= 0) {
      TPS_TRY(st->prefetch_mb(mb));
      for (int l = 0; l < p.L; ++l) TPS_HIP(hipStreamWaitEvent(st->cs, st->ready_ev[mb][l], 0));
    }
  }
  // segment granularity (one micro-batch, checked above): the whole replay
  // runs before the first layer backward, each layer on its own window entry
  // (with streamed weights a replay may evict the entry of another layer, so
  // no entry is bound across it)
  if (p.granularity == TPS_GRAN_SEGMENT) {
    for (int r = 0; r < p.L; ++r) {
      if (!p.replay_ops[r]) continue;
      int er = -1;
      TPS_TRY(st->ensure_layer(r, false, &er));
      void* yl = (r == p.L - 1) ? nullptr : st->tensor(r + 1, TPS_T_X, mb0, true);
      TPS_TRY(st->fwd_layer(r, mb0, st->params_of(r, &er), yl, p.replay_ops[r], true, true));
      TPS_TRY(st->touch(er));
      ++st->stats.replays;
    }
  }
  if (p.grp_n > 0 && n > 1 && n <= p.grp_n && p.granularity == TPS_GRAN_LAYER) {
    // Batched weight gradients: the running input gradients of the group
    // alternate between two slot buffers by layer (layer 0 writes the
    // caller's dx), the layer's operands stay in the group's slots, and each
    // weight-gradient product runs once per layer over the n micro-batches.
    int yin = 0;
    for (int i = 0; i < n; ++i)
      TPS_HIP(hipMemcpyAsync(st->grp_slot(p.work.grp_y[0], p.tbytes[TPS_T_X], i), dy[i], p.tbytes[TPS_T_X],
                             hipMemcpyDeviceToDevice, st->cs));
    for (int l = p.L - 1; l >= 0; --l) {
      int e = -1;
      TPS_TRY(st->ensure_layer(l, true, &e));
      TPS_TRY(st->prefetch_layer(l - 1));
      const char* W = st->params_of(l, &e);
      const bool bl = st->layer_batchable(l);
      const bool fresh = st->grads_fresh[l] != 0;   // the layer backwards below clear it
      for (int i = 0; i < n; ++i) {
        const int mb = mb0 + i;
        st->grp_i = bl ? i : -1;
        if (p.replay_ops[l]) {
          TPS_TRY(st->fwd_layer(l, mb, W, nullptr, p.replay_ops[l], true, true));
          ++st->stats.replays;
        }
        const void* in = st->grp_slot(p.work.grp_y[yin], p.tbytes[TPS_T_X], i);
        void* out = l == 0 ? dx[i] : st->grp_slot(p.work.grp_y[yin ^ 1], p.tbytes[TPS_T_X], i);
        const int rc = st->bwd_layer(l, mb, W, st->wt_of(l, e), st->grads_of(l, e), in, out, 0, false, bl ? i : -1);
        st->grp_i = -1;
        TPS_TRY(rc);
      }
      if (bl) TPS_TRY(st->batched_wgrad(l, st->grads_of(l, e), n, fresh, yin));
      TPS_TRY(st->touch(e));
      TPS_TRY(st->opt_after_backward(l, n));
      yin ^= 1;
    }
  } else {
  char* gA = st->work(p.work.g[0]);
  for (int l = p.L - 1; l >= 0; --l) {
    int e = -1;
    TPS_TRY(st->ensure_layer(l, true, &e));
    TPS_TRY(st->prefetch_layer(l - 1));
    const char* W = st->params_of(l, &e);
    for (int i = 0; i < n; ++i) {
      const int mb = mb0 + i;
      if (p.granularity == TPS_GRAN_LAYER && p.replay_ops[l]) {
        TPS_TRY(st->fwd_layer(l, mb, W, nullptr, p.replay_ops[l], true, true));
        ++st->stats.replays;
      }
      // the running gradient of micro-batch i lives in dx[i] between layers
      const void* in = (l == p.L - 1) ? dy[i] : dx[i];
      TPS_TRY(st->bwd_layer(l, mb, W, st->wt_of(l, e), st->grads_of(l, e), in, gA, 0, false));
      TPS_HIP(hipMemcpyAsync(dx[i], gA, p.tbytes[TPS_T_X], hipMemcpyDeviceToDevice, st->cs));
    }
    TPS_TRY(st->touch(e));
    TPS_TRY(st->opt_after_backward(l, n));
  }
  }
  for (int i = 0; i < n; ++i) {
    const int mb = mb0 + i;
    if (p.oslot_bytes) TPS_TRY(st->release_oslot(p.oslot_b[mb], st->cs));
    TPS_TRY(st->poison_after_backward(mb));
    st->b_done[mb] = 1;
    ++st->cursor;
  }
  st->stats.ops_done = st->cursor;
  if (st->cursor == (int)p.op_kind.size()) return st->flush_all_grads();
  return TPS_OK;
}

extern "C" int tps_stage_sync(tps_stage* st) {
  clear_error();
  if (!st) return set_error(TPS_EINVAL, "null stage");
  TPS_HIP(hipStreamSynchronize(st->cs));
  if (st->xs) TPS_HIP(hipStreamSynchronize(st->xs));
  if (st->ps && st->ps != st->xs) TPS_HIP(hipStreamSynchronize(st->ps));
  if (st->gs) TPS_HIP(hipStreamSynchronize(st->gs));
  if (st->rs) TPS_HIP(hipStreamSynchronize(st->rs));
  return st->wait_all_updates();
}

extern "C" int tps_stage_set_optimizer(tps_stage* st, const tps_adamw* opt, float* const* master, float* const* m,
                                       float* const* v, int32_t first_step, int32_t n_threads) {
  return tps_stage_set_optimizer_split(st, opt, master, m, v, nullptr, 0, first_step, n_threads);
}

extern "C" int tps_stage_set_optimizer_split(tps_stage* st, const tps_adamw* opt, float* const* master,
                                             float* const* m, float* const* v, void* const* dparams, int32_t n_device,
                                             int32_t first_step, int32_t n_threads) {
  clear_error();
  if (!st || !opt || !master || !m || !v) return set_error(TPS_EINVAL, "tps_stage_set_optimizer: null argument");
  if (n_device < 0 || n_device > st->p.L) return set_error(TPS_EINVAL, "tps_stage_set_optimizer: n_device out of range");
  if (n_device > 0 && !dparams) return set_error(TPS_EINVAL, "tps_stage_set_optimizer: null device parameter blocks");
  for (int l = 0; l < n_device; ++l) {
    if (!dparams[l]) return set_error(TPS_EINVAL, "tps_stage_set_optimizer: null device parameter block");
    // the device update reads and writes 16-byte groups of the f32 blocks
    if (((uintptr_t)master[l] | (uintptr_t)m[l] | (uintptr_t)v[l]) & 15u)
      return set_error(TPS_EINVAL, "tps_stage_set_optimizer: device blocks must be 16-byte aligned");
  }
  const Plan& p = st->p;
  if (p.weights != TPS_W_STREAM) return set_error(TPS_EINVAL, "tps_stage_set_optimizer: needs streamed weights");
  if (st->hopt.on) return set_error(TPS_ESTATE, "tps_stage_set_optimizer: already set");
  if (st->in_iteration && st->cursor != 0 && st->cursor < (int)p.op_kind.size())
    return set_error(TPS_ESTATE, "tps_stage_set_optimizer: inside an iteration");
  if (first_step < 1) return set_error(TPS_EINVAL, "tps_stage_set_optimizer: first_step must be >= 1");
  if (!(opt->lr >= 0.f && opt->beta1 >= 0.f && opt->beta1 < 1.f && opt->beta2 >= 0.f && opt->beta2 < 1.f &&
        opt->eps >= 0.f && opt->weight_decay >= 0.f))
    return set_error(TPS_EINVAL, "tps_stage_set_optimizer: hyper-parameters out of range");
  for (int l = 0; l < p.L; ++l)
    if (!master[l] || !m[l] || !v[l]) return set_error(TPS_EINVAL, "tps_stage_set_optimizer: null layer block");
  auto& h = st->hopt;
  h.hp = *opt;
  h.threads = n_threads;
  h.master.assign(master, master + p.L);
  h.m.assign(m, m + p.L);
  h.v.assign(v, v + p.L);
  h.step.assign(p.L, first_step);
  h.bpass.assign(p.L, 0);
  h.pending.assign(p.L, 0);
  h.final_ev.assign(p.L, nullptr);
  for (auto& e : h.final_ev) TPS_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  h.n_dev = n_device;
  h.dparams.assign(p.L, nullptr);
  for (int l = 0; l < n_device; ++l) h.dparams[l] = dparams[l];
  h.dev_ev.assign(p.L, nullptr);
  h.dev_ev_valid.assign(p.L, 0);
  for (int l = 0; l < n_device; ++l)
    TPS_HIP(hipEventCreateWithFlags(&h.dev_ev[l], hipEventDisableTiming | hipEventDisableSystemFence));
  h.on = true;
  h.worker = std::thread([st] { st->opt_worker(); });
  return TPS_OK;
}

// Bounded wait: polls every stream of the stage until all are idle, a
// stream reports an error, or the deadline passes.
extern "C" int tps_stage_sync_for(tps_stage* st, double timeout_ms) {
  clear_error();
  if (!st) return set_error(TPS_EINVAL, "null stage");
  if (!(timeout_ms >= 0.0)) return set_error(TPS_EINVAL, "tps_stage_sync_for: negative or NaN timeout");
  struct Named {
    hipStream_t s;
    const char* name;
  };
  std::vector<Named> streams = {{st->cs, "compute"}};
  if (st->gs && st->gs != st->cs) streams.push_back({st->gs, "parameter-gradient"});
  if (st->rs) streams.push_back({st->rs, "replay"});
  if (st->xs) streams.push_back({st->xs, "device-to-host copy"});
  if (st->ps && st->ps != st->xs) streams.push_back({st->ps, "host-to-device copy"});
  const auto t0 = std::chrono::steady_clock::now();
  for (;;) {
    const char* busy = nullptr;
    for (const Named& n : streams) {
      const hipError_t e = hipStreamQuery(n.s);
      if (e == hipErrorNotReady) {
        if (!busy) busy = n.name;
        continue;
      }
      if (e != hipSuccess) return check_hip(e, "tps_stage_sync_for");
    }
    if (!busy) return TPS_OK;
    const double ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    if (ms >= timeout_ms)
      return set_error(TPS_ETIMEOUT, std::string("tps_stage_sync_for: the ") + busy + " stream still has work after " +
                                         std::to_string(timeout_ms) + " ms");
    std::this_thread::sleep_for(std::chrono::microseconds(50));
  }
}

extern "C" int tps_stage_stats(const tps_stage* st, tps_stats* out) {
  clear_error();
  if (!st || !out) return set_error(TPS_EINVAL, "null argument");
  // the host optimizer's thread adds its timings under its lock
  std::lock_guard<std::mutex> lock(const_cast<tps_stage*>(st)->hopt.mu);
  *out = st->stats;
  return TPS_OK;
}

extern "C" int tps_stage_time_kernels(tps_stage* st, const char* prefix) {
  clear_error();
  if (!st) return set_error(TPS_EINVAL, "null stage");
  TPS_HIP(hipStreamSynchronize(st->cs));
  TPS_TRY(st->kresolve());
  st->tagg.clear();
  st->timing = prefix != nullptr;
  st->tprefix = prefix ? prefix : "";
  return TPS_OK;
}

extern "C" int tps_stage_kernel_times(tps_stage* st, tps_kernel_time* out, int max, int* n_out) {
  clear_error();
  if (!st || (!out && max > 0)) return set_error(TPS_EINVAL, "null argument");
  TPS_HIP(hipStreamSynchronize(st->cs));
  TPS_TRY(st->kresolve());
  int n = 0;
  for (auto& kv : st->tagg) {
    if (n < max) out[n] = kv.second;
    ++n;
  }
  if (n_out) *n_out = n;
  return TPS_OK;
}

extern "C" int tps_stage_destroy(tps_stage* st) {
  clear_error();
  if (!st) return TPS_OK;
  if (st->hopt.worker.joinable()) {
    {
      std::lock_guard<std::mutex> lock(st->hopt.mu);
      st->hopt.stop = true;
    }
    st->hopt.cv.notify_all();
    st->hopt.worker.join();
  }
  for (auto e : st->hopt.final_ev)
    if (e) (void)hipEventDestroy(e);
  for (auto e : st->hopt.dev_ev)
    if (e) (void)hipEventDestroy(e);
  if (st->cs) (void)hipStreamSynchronize(st->cs);
  if (st->xs) (void)hipStreamSynchronize(st->xs);
  if (st->ps && st->ps != st->xs) (void)hipStreamSynchronize(st->ps);
  if (st->gs && st->gs != st->cs) {
    (void)hipStreamSynchronize(st->gs);
    (void)hipStreamDestroy(st->gs);
  }
  if (st->own_xs) (void)hipStreamDestroy(st->xs);
  if (st->own_ps) (void)hipStreamDestroy(st->ps);
  if (st->ev_fork) (void)hipEventDestroy(st->ev_fork);
  if (st->ev_join) (void)hipEventDestroy(st->ev_join);
  for (auto e : st->ev_gs)
    if (e) (void)hipEventDestroy(e);
  if (st->rs) {
    (void)hipStreamSynchronize(st->rs);
    (void)hipStreamDestroy(st->rs);
  }
  if (st->ev_rfork) (void)hipEventDestroy(st->ev_rfork);
  for (auto e : st->ev_replay)
    if (e) (void)hipEventDestroy(e);
  if (st->ev_tmp) (void)hipEventDestroy(st->ev_tmp);
  for (auto* v : {&st->oslot_ev, &st->offloaded_ev, &st->hslot_read_ev, &st->lgrads_out_ev})
    for (auto& s : *v)
      if (s.ev) (void)hipEventDestroy(s.ev);
  for (auto& v : st->ready_ev)
    for (auto e : v)
      if (e) (void)hipEventDestroy(e);
  for (auto& r : st->tpending) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : st->tpool) (void)hipEventDestroy(e);
  for (auto& w : st->win) {
    if (w.param_ready.ev) (void)hipEventDestroy(w.param_ready.ev);
    if (w.last_use.ev) (void)hipEventDestroy(w.last_use.ev);
    if (w.grads_out.ev) (void)hipEventDestroy(w.grads_out.ev);
  }
  delete st;
  return TPS_OK;
}

extern "C" int tps_host_alloc(uint64_t bytes, void** out) {
  clear_error();
  if (!out) return set_error(TPS_EINVAL, "null argument");
  *out = nullptr;
  if (bytes == 0) return TPS_OK;
  const hipError_t e = hipHostMalloc(out, bytes, hipHostMallocDefault);
  if (e != hipSuccess) {
    *out = nullptr;
    (void)hipGetLastError();
    return set_error(TPS_ENOMEM, "cannot pin " + std::to_string(bytes) + " bytes of host memory: " +
                                     hipGetErrorString(e));
  }
  return TPS_OK;
}

extern "C" int tps_host_free(void* p) {
  clear_error();
  if (!p) return TPS_OK;
  TPS_HIP(hipHostFree(p));
  return TPS_OK;
}
