// Stage planner: host-only (no HIP calls), so tps_plan() runs without a GPU.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/tpstage.h"

namespace tps {

// Forward operators of one layer, in execution order.
enum FwdOp { OP_LN1 = 0, OP_QKV, OP_ATTN, OP_OPROJ, OP_LN2, OP_FC1, OP_GELU, OP_FC2, OP_COUNT };

constexpr uint64_t kNone = ~0ull;

struct Plan {
  // shape
  int L = 0, h = 0, nh = 0, d = 0, f = 0, s = 0, b = 0, M = 0, T = 0;
  // layer kind: LLAMA (RMSNorm, rotary embedding, nkv key/value heads, SwiGLU,
  // no biases) or GPT; qw: width of the packed qkv tensor, uw: of u
  bool llama = false;
  int nkv = 0;
  float rope_base = 10000.f;
  int64_t qw = 0, uw = 0;
  // shape of each packed parameter ([rows][cols]; 0 x 0 when absent)
  int64_t prow[TPS_P_COUNT] = {}, pcol[TPS_P_COUNT] = {};
  int dtype = TPS_BF16, esize = 2;
  float eps = 1e-5f;
  int weights = TPS_W_RESIDENT, window = 2, granularity = TPS_GRAN_SEGMENT, lookahead = 1;
  std::vector<uint8_t> policy;        // [L][TPS_T_COUNT]
  uint64_t offload_mask = 0;

  // order
  std::vector<int> op_kind, op_mb;    // planned F/B order
  std::vector<int> pos_f, pos_b;      // op index of F(mb), B(mb)

  // sizes
  uint64_t tbytes[TPS_T_COUNT] = {};  // bytes of each tensor of one (layer, mb)
  uint64_t poff[TPS_P_COUNT] = {}, pbytes = 0;   // packed parameter block
  uint64_t goff[TPS_P_COUNT] = {}, gbytes = 0;   // packed f32 gradient block
  // quantized host parameter block (weights_quant == TPS_Q_FP8_ROW): codes or
  // storage-dtype vectors at qoff, f32 row scales of the four matrices at qsoff
  int quant = TPS_Q_NONE;
  bool wgrad_inline = false;   // parameter-gradient kernels on the compute stream
  uint64_t qoff[TPS_P_COUNT] = {}, qsoff[4] = {}, qbytes = 0;
  uint64_t hpbytes = 0;   // bytes of one host parameter block (pbytes or qbytes)

  // Checkpoint slots of one micro-batch, in two parts:
  //  - resident part: KEEP tensors of every layer, held from F(mb) to B(mb);
  //  - offload part: OFFLOAD tensors of every layer.  Held from F(mb) to B(mb)
  //    for micro-batches that are not offloaded; for offloaded ones held
  //    during F(mb) (until the copies to host finish) and again from the
  //    prefetch to the end of B(mb).  Host slots use the same layout.
  std::vector<uint64_t> kslot_off;    // [L][T_COUNT], kNone if not KEEP
  uint64_t kslot_bytes = 0;
  int n_kslots = 0;
  std::vector<int> kslot;             // [M]
  std::vector<uint64_t> oslot_off;    // [L][T_COUNT], kNone if not OFFLOAD
  uint64_t oslot_bytes = 0;
  int n_oslots = 0;
  std::vector<int> oslot_f, oslot_b;  // [M]
  int max_inflight = 0;
  int n_host_slots = 0;
  std::vector<int> host_slot;         // [M], -1 if the mb is not offloaded
  std::vector<std::vector<int>> prefetch_at;  // [n_ops]: mbs brought back before op p

  // recompute: replay buffer and per-layer replay program
  std::vector<uint64_t> replay_off;   // [L][T_COUNT], kNone if not recomputed
  uint64_t replay_bytes = 0;
  std::vector<uint32_t> replay_ops;   // [L] bit mask over FwdOp
  int n_replay_layers = 0;

  // backward working buffers (offsets inside the work region): the running
  // input gradient between layers (g, rotating), the layer's intermediate
  // gradients (dx1, du, dqkv: one set per layer parity when defer_join),
  // the attention output projection's input gradient (t1) and the
  // attention backward's row dot products (dvec)
  // (LLAMA: dg, the gradient of the SwiGLU output before its backward;
  // kvws, the per-query-head key/value gradients of grouped attention; rope,
  // the rotation table; zbias, a zero vector standing in for the absent
  // biases in the residual epilogues)
  struct Work {
    uint64_t g[3], dx1[2], du[2], dqkv[2], t1, dvec;
    uint64_t dg, kvws, rope, zbias;
    // batched weight gradients of backward groups (group_wgrad): per
    // micro-batch slots [grp_n][T, width] of the layer's a, o, c, g (the
    // activation operands), du, dx1, dqkv (the gradient operands) and the
    // running input gradient (two, alternating by layer)
    uint64_t grp_act[4], grp_du, grp_dx1, grp_dqkv, grp_y[2];
  } work{};
  int grp_n = 0;   // largest group the slots hold (0: no batched weight gradients)
  uint64_t work_bytes = 0;
  // the parameter-gradient kernels of a layer backward may still run while
  // the next layer's input-gradient chain starts; the two streams join once
  // per micro-batch (resident weights, and no replay between layer
  // backwards, whose buffers the lagging kernels could still be reading)
  bool defer_join = false;
  // no layer's replay reads another layer's replayed output (every layer
  // input is kept or offloaded): the segment replay may run in any layer order
  bool replay_independent = false;

  // per-layer f32 partial sums of the bias and LayerNorm parameter gradients:
  // [segments][bpart_cols] with column ranges (bpc[]) for b_qkv, b_o, b_1,
  // b_2, beta1, gamma1, beta2, gamma2; summed over segments into the grads
  // when those are handed over
  enum { BP_QKV, BP_O, BP_1, BP_2, BP_BE1, BP_G1, BP_BE2, BP_G2, BP_COUNT };
  int64_t bpc[BP_COUNT + 1] = {};
  int bpart_segs = 0;
  uint64_t bpart_bytes = 0;   // one layer's block

  // transposed weight matrices (B operands of the input-gradient GEMMs):
  // Wqkv^T [h, 3h], Wo^T [h, h], W1^T [h, f], W2^T [f, h] per layer
  uint64_t wtoff[4] = {}, wt_bytes = 0;
  uint64_t wt_region = 0;   // L blocks (resident) or window blocks (streamed)

  // streamed weights window
  uint64_t wwin_bytes = 0;

  // arena
  uint64_t off_wt = 0;
  uint64_t off_kslots = 0, off_oslots = 0, off_replay = 0, off_work = 0, off_wwin = 0, off_bpart = 0;
  uint64_t arena_bytes = 0, host_bytes = 0;

  // accounting
  double fwd_flops = 0, bwd_flops = 0, recompute_flops = 0;
  uint64_t h2d_bytes = 0, d2h_bytes = 0;
  uint64_t keep_all_bytes = 0, predicted_peak = 0;

  int mode(int layer, int t, int mb) const {
    const int p = policy[layer * TPS_T_COUNT + t];
    if (p == TPS_OFFLOAD && !((offload_mask >> mb) & 1ull)) return TPS_KEEP;
    return p;
  }
  int pol(int layer, int t) const { return policy[layer * TPS_T_COUNT + t]; }
  bool offloaded(int mb) const { return host_slot[mb] >= 0; }
};

// Builds the plan; returns TPS_OK or an error code (message via set_error).
int make_plan(const tps_config* cfg, Plan* out);

// Algorithmic flops of one forward operator for one (layer, mb).
double op_flops(const Plan& p, int op);

void fill_plan_info(const Plan& p, tps_plan_info* info);

// f32 coefficients of one AdamW step (step >= 1), computed once per layer
// update in double and rounded to f32: lr_c = lr / (1 - b1^step),
// inv_bc2_sqrt = 1 / sqrt(1 - b2^step), wd_c = lr wd.  The host update and the
// device update take the same values.
struct AdamwCoef {
  float b1, b2, eps, lr_c, inv_bc2_sqrt, wd_c;
};
AdamwCoef adamw_coef(const tps_adamw& opt, int32_t step);

// One host AdamW step of a layer and its parameter block for the device
// (tps_host_adamw_layer, on an existing plan).
int host_adamw(const Plan& p, const tps_adamw* opt, int32_t step, float* master, float* m, float* v,
               const float* grad, void* params_out, int32_t quant, int32_t n_threads);

}  // namespace tps
