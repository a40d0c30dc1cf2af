// Stage planner (host only): op order, policy closure and replay program,
// checkpoint-slot assignment over the order, arena layout, offload victim
// selection and byte / flop accounting.
#include "planner.h"

#include <algorithm>
#include <functional>
#include <numeric>
#include <queue>
#include <set>

#include "errors.h"
#include "ws.h"

namespace tps {

namespace {

uint64_t align256(uint64_t x) { return (x + 255) & ~255ull; }

int inval(const std::string& m) { return set_error(TPS_EINVAL, "config: " + m); }

// Smallest free slot index first, so the assignment is a pure function of the
// order.
struct SlotPool {
  std::set<int> free_;
  int count = 0;
  int acquire() {
    if (free_.empty()) return count++;
    const int s = *free_.begin();
    free_.erase(free_.begin());
    return s;
  }
  void release(int s) { free_.insert(s); }
};

// Slots that become free at a time (the end of a copy).  acquire(t) takes
// the smallest index free by t; acquire(t, latest, &when) may also wait for
// the slot that frees first if that happens by `latest` (when: the time the
// slot is taken); otherwise a new slot.
struct TimedSlotPool {
  std::vector<double> free_at;   // < 0: in use
  int count() const { return (int)free_at.size(); }
  int acquire(double t, double latest = -1, double* when = nullptr) {
    if (when) *when = t;
    int best = -1;
    for (size_t s = 0; s < free_at.size(); ++s) {
      if (free_at[s] < 0) continue;
      if (free_at[s] <= t) {
        best = (int)s;
        break;
      }
      if (free_at[s] <= latest && (best < 0 || free_at[s] < free_at[best])) best = (int)s;
    }
    if (best < 0) {
      free_at.push_back(-1);
      return (int)free_at.size() - 1;
    }
    if (when) *when = std::max(t, free_at[best]);
    free_at[best] = -1;
    return best;
  }
  void release(int s, double t) { free_at[s] = t; }
};

}  // namespace

double op_flops(const Plan& p, int op) {
  const double T = p.T, h = p.h, f = p.f;
  switch (op) {
    case OP_QKV: return 2.0 * T * h * (double)p.qw;
    case OP_ATTN: return 2.0 * p.b * h * (double)p.s * (p.s + 1);
    case OP_OPROJ: return 2.0 * T * h * h;
    case OP_FC1: return 2.0 * T * h * (double)p.uw;
    case OP_FC2: return 2.0 * T * f * h;
    default: return 0.0;
  }
}

static int build_order(const tps_config* c, Plan& p) {
  const int M = p.M;
  if (c->n_ops == 0) {
    const int W = (c->inflight <= 0 || c->inflight > M) ? M : c->inflight;
    for (int i = 0; i < W; ++i) { p.op_kind.push_back(TPS_OP_F); p.op_mb.push_back(i); }
    int next = W;
    for (int i = 0; i < M; ++i) {
      p.op_kind.push_back(TPS_OP_B); p.op_mb.push_back(i);
      if (next < M) { p.op_kind.push_back(TPS_OP_F); p.op_mb.push_back(next++); }
    }
  } else {
    if (c->n_ops != 2 * M || c->ops == nullptr) return inval("ops must list F and B of every micro-batch once");
    for (int i = 0; i < c->n_ops; ++i) {
      p.op_kind.push_back(c->ops[2 * i]);
      p.op_mb.push_back(c->ops[2 * i + 1]);
    }
  }
  p.pos_f.assign(M, -1);
  p.pos_b.assign(M, -1);
  for (size_t i = 0; i < p.op_kind.size(); ++i) {
    const int k = p.op_kind[i], mb = p.op_mb[i];
    if (mb < 0 || mb >= M || (k != TPS_OP_F && k != TPS_OP_B)) return inval("ops entry out of range");
    int& slot = (k == TPS_OP_F) ? p.pos_f[mb] : p.pos_b[mb];
    if (slot >= 0) return inval("ops lists a task twice");
    slot = (int)i;
  }
  for (int mb = 0; mb < M; ++mb)
    if (p.pos_f[mb] < 0 || p.pos_b[mb] < 0 || p.pos_b[mb] < p.pos_f[mb])
      return inval("ops: every B(mb) must follow its F(mb)");
  return TPS_OK;
}

// Replay program of each layer: the forward operators whose outputs include a
// recomputed tensor, closed over their recomputed inputs.  A recomputed layer
// input X(l) makes layer l-1 replay through FC2.
static void build_replay(Plan& p) {
  p.replay_ops.assign(p.L, 0);
  std::vector<char> need_y(p.L, 0);
  for (int l = p.L - 1; l >= 0; --l) {
    bool avail[TPS_T_COUNT], made[TPS_T_COUNT] = {};
    for (int t = 0; t < TPS_T_COUNT; ++t) avail[t] = p.pol(l, t) != TPS_RECOMPUTE;
    uint32_t ops = 0;
    std::function<void(int)> want = [&](int t) {
      if (avail[t] || made[t]) return;
      made[t] = true;
      switch (t) {
        case TPS_T_X: if (l > 0) need_y[l - 1] = 1; break;
        case TPS_T_A: case TPS_T_LN1:
          made[TPS_T_A] = made[TPS_T_LN1] = true; want(TPS_T_X); ops |= 1u << OP_LN1; break;
        case TPS_T_QKV: want(TPS_T_A); ops |= 1u << OP_QKV; break;
        case TPS_T_O: case TPS_T_LSE:
          made[TPS_T_O] = made[TPS_T_LSE] = true; want(TPS_T_QKV); ops |= 1u << OP_ATTN; break;
        case TPS_T_X1: want(TPS_T_O); want(TPS_T_X); ops |= 1u << OP_OPROJ; break;
        case TPS_T_C: case TPS_T_LN2:
          made[TPS_T_C] = made[TPS_T_LN2] = true; want(TPS_T_X1); ops |= 1u << OP_LN2; break;
        case TPS_T_U:
          made[TPS_T_G] = true; want(TPS_T_C); ops |= 1u << OP_FC1; break;
        case TPS_T_G:
          if (avail[TPS_T_U]) { ops |= 1u << OP_GELU; }
          else { made[TPS_T_G] = false; want(TPS_T_U); }
          break;
      }
    };
    for (int t = 0; t < TPS_T_COUNT; ++t)
      if (!avail[t]) want(t);
    if (need_y[l]) {
      want(TPS_T_G);
      want(TPS_T_X1);
      ops |= 1u << OP_FC2;
    }
    p.replay_ops[l] = ops;
  }
  p.n_replay_layers = 0;
  for (int l = 0; l < p.L; ++l) p.n_replay_layers += p.replay_ops[l] != 0;
}

// Compute-time model for victim choice: F and B costs from flops at the hinted
// rate; each offloaded micro-batch sends its bytes down after F and back before
// B over one link per direction.  Returns the simulated iteration time.
static double simulate_offload(const Plan& p, const std::vector<char>& victim, double tF, double tB, double tc) {
  double t = 0, d2h_free = 0, h2d_free = 0;
  std::vector<double> d2h_end(p.M, 0), h2d_end(p.M, 0);
  const int nops = (int)p.op_kind.size();
  for (int i = 0; i < nops; ++i) {
    for (int mb = 0; mb < p.M; ++mb) {
      if (!victim[mb]) continue;
      const int at = std::max(p.pos_f[mb] + 1, p.pos_b[mb] - p.lookahead);
      if (at == i) {
        const double st = std::max({t, h2d_free, d2h_end[mb]});
        h2d_end[mb] = st + tc;
        h2d_free = h2d_end[mb];
      }
    }
    const int mb = p.op_mb[i];
    if (p.op_kind[i] == TPS_OP_F) {
      t += tF;
      if (victim[mb]) {
        const double st = std::max(t, d2h_free);
        d2h_end[mb] = st + tc;
        d2h_free = d2h_end[mb];
      }
    } else {
      if (victim[mb]) t = std::max(t, h2d_end[mb]);
      t += tB;
    }
  }
  return t;
}

// Slot and host-slot assignment along the order for p.offload_mask, timed
// with the model of the order (tF, tB: one micro-batch's forward and
// backward, tc: one micro-batch's offload copy): an offloaded micro-batch's
// staging slot is free once its device -> host copy (queued behind earlier
// ones) is done, a host slot once the prefetch out of it is done, so a
// forward never waits on a copy for its slot; the slot count is what the
// overlap costs in memory.  Returns the number of staging slots.
static int assign_slots(Plan& p, double tF, double tB, double tc) {
  p.host_slot.assign(p.M, -1);
  p.kslot.assign(p.M, -1);
  p.oslot_f.assign(p.M, -1);
  p.oslot_b.assign(p.M, -1);
  p.prefetch_at.assign(p.op_kind.size(), {});
  for (int mb = 0; mb < p.M; ++mb)
    if ((p.offload_mask >> mb) & 1ull) {
      const int at = std::max(p.pos_f[mb] + 1, p.pos_b[mb] - p.lookahead);
      p.prefetch_at[at].push_back(mb);
    }
  SlotPool kpool;
  TimedSlotPool opool, hpool;
  int inflight = 0;
  double t = 0, d2h_free = 0, h2d_free = 0;
  std::vector<double> d2h_end(p.M, 0), h2d_end(p.M, 0);
  for (size_t i = 0; i < p.op_kind.size(); ++i) {
    for (int mb : p.prefetch_at[i]) {
      // a prefetch may wait for a slot up to one copy time (a forward may not)
      double st = std::max({t, h2d_free, d2h_end[mb]});
      p.oslot_b[mb] = opool.acquire(st, st + tc, &st);
      h2d_end[mb] = h2d_free = st + tc;
      hpool.release(p.host_slot[mb], h2d_end[mb]);
    }
    const int mb = p.op_mb[i];
    const bool off = (p.offload_mask >> mb) & 1ull;
    if (p.op_kind[i] == TPS_OP_F) {
      ++inflight;
      p.max_inflight = std::max(p.max_inflight, inflight);
      p.kslot[mb] = kpool.acquire();
      p.oslot_f[mb] = opool.acquire(t);
      t += tF;
      if (off) {
        // the copy to host queues behind earlier ones and waits for a host slot
        double st = std::max(t, d2h_free);
        p.host_slot[mb] = hpool.acquire(st, st + tc, &st);
        d2h_end[mb] = d2h_free = st + tc;
        opool.release(p.oslot_f[mb], d2h_end[mb]);
      } else {
        p.oslot_b[mb] = p.oslot_f[mb];
      }
    } else {
      if (off) t = std::max(t, h2d_end[mb]);
      t += tB;
      --inflight;
      kpool.release(p.kslot[mb]);
      opool.release(p.oslot_b[mb], t);
    }
  }
  p.n_kslots = p.kslot_bytes ? kpool.count : 0;
  p.n_oslots = p.oslot_bytes ? opool.count() : 0;
  p.n_host_slots = p.oslot_bytes ? hpool.count() : 0;
  return opool.count();
}

int make_plan(const tps_config* c, Plan* out) {
  if (!c || !out) return inval("null argument");
  if (c->abi_version != TPS_ABI_VERSION) return inval("abi_version mismatch");
  Plan p;
  p.L = c->n_layers; p.h = c->hidden; p.nh = c->n_heads; p.f = c->mlp;
  p.s = c->seq; p.b = c->micro_batch; p.M = c->n_micro;
  p.dtype = c->dtype; p.eps = c->ln_eps;
  if (p.L < 1 || p.L > 4096) return inval("n_layers");
  if (p.h <= 0 || p.nh <= 0 || p.h % p.nh) return inval("hidden must be a multiple of n_heads");
  p.d = p.h / p.nh;
  if (p.d != 64 && p.d != 128) return inval("head dim hidden/n_heads must be 64 or 128");
  if (p.h % 8 || p.f <= 0 || p.f % 8) return inval("hidden and mlp must be positive multiples of 8");
  if (p.h > 16384) return inval("hidden must be <= 16384");
  if (p.s < 1 || p.b < 1) return inval("seq and micro_batch must be >= 1");
  if (p.M < 1 || p.M > TPS_MAX_MICRO) return inval("n_micro must be in 1..64");
  if ((int64_t)p.b * p.s > (1ll << 30)) return inval("micro_batch * seq too large");
  if (p.dtype != TPS_F32 && p.dtype != TPS_BF16) return inval("dtype");
  if (!(p.eps >= 0.f)) return inval("ln_eps must be >= 0");
  p.esize = p.dtype == TPS_BF16 ? 2 : 4;
  p.T = p.b * p.s;
  p.weights = c->weights;
  if (p.weights != TPS_W_RESIDENT && p.weights != TPS_W_STREAM) return inval("weights");
  p.window = c->window;
  // a window of two serves a single layer too (one entry stays unused)
  if (p.weights == TPS_W_STREAM && (p.window < 2 || p.window > (p.L < 2 ? 2 : p.L)))
    return inval("window must be in 2..max(2, n_layers)");
  p.granularity = c->recompute_granularity;
  if (p.granularity != TPS_GRAN_LAYER && p.granularity != TPS_GRAN_SEGMENT) return inval("recompute_granularity");
  p.lookahead = c->lookahead;
  if (p.lookahead < 1) return inval("lookahead must be >= 1");
  if (c->wgrad_stream < TPS_WGRAD_AUTO || c->wgrad_stream > TPS_WGRAD_INLINE) return inval("wgrad_stream");
  if (c->group_wgrad != 0 && c->group_wgrad != 1) return inval("group_wgrad");
  // same-device A/B of the two arrangements: inline was 2-3% faster at 4096
  // and 8192 tokens per micro-batch, 10% slower at 2048
  p.wgrad_inline = c->wgrad_stream == TPS_WGRAD_INLINE || (c->wgrad_stream == TPS_WGRAD_AUTO && p.T >= 4096);
  if (c->arch != TPS_ARCH_GPT && c->arch != TPS_ARCH_LLAMA) return inval("arch");
  p.llama = c->arch == TPS_ARCH_LLAMA;
  p.nkv = c->n_kv_heads ? c->n_kv_heads : p.nh;
  if (p.llama) {
    if (p.dtype != TPS_BF16 || p.d != 128) return inval("LLAMA layers need bf16 storage and head dim 128");
    if (p.nkv < 1 || p.nkv > p.nh || p.nh % p.nkv) return inval("n_kv_heads must divide n_heads");
    p.rope_base = c->rope_base == 0.f ? 10000.f : c->rope_base;
    if (!(p.rope_base > 1.f)) return inval("rope_base must be > 1");
  } else if (p.nkv != p.nh) {
    return inval("n_kv_heads applies to LLAMA layers only");
  }
  p.qw = (int64_t)(p.nh + 2 * p.nkv) * p.d;
  p.uw = p.llama ? 2 * (int64_t)p.f : p.f;
  {
    const int64_t H = p.h, F = p.f;
    const int64_t gpt_r[TPS_P_COUNT] = {3 * H, 1, H, 1, F, 1, H, 1, 1, 1, 1, 1};
    const int64_t gpt_c[TPS_P_COUNT] = {H, 3 * H, H, H, H, F, F, H, H, H, H, H};
    const int64_t lla_r[TPS_P_COUNT] = {p.qw, 0, H, 0, 2 * F, 0, H, 0, 1, 0, 1, 0};
    const int64_t lla_c[TPS_P_COUNT] = {H, 0, H, 0, H, 0, F, 0, H, 0, H, 0};
    for (int i = 0; i < TPS_P_COUNT; ++i) {
      p.prow[i] = p.llama ? lla_r[i] : gpt_r[i];
      p.pcol[i] = p.llama ? lla_c[i] : gpt_c[i];
    }
  }
  p.quant = c->weights_quant;
  if (p.quant != TPS_Q_NONE && p.quant != TPS_Q_FP8_ROW) return inval("weights_quant");
  if (p.quant == TPS_Q_FP8_ROW && (p.weights != TPS_W_STREAM || p.dtype != TPS_BF16))
    return inval("quantized weight reload needs streamed bf16 weights");

  // policy
  p.policy.assign((size_t)p.L * TPS_T_COUNT, TPS_KEEP);
  if (c->policy) {
    for (size_t i = 0; i < p.policy.size(); ++i) {
      if (c->policy[i] > TPS_OFFLOAD) return inval("policy value");
      p.policy[i] = c->policy[i];
    }
  }
  if (p.pol(0, TPS_T_X) == TPS_RECOMPUTE) return inval("the stage input X of layer 0 cannot be recomputed");
  if (p.granularity == TPS_GRAN_LAYER)
    for (int l = 0; l < p.L; ++l)
      if (p.pol(l, TPS_T_X) == TPS_RECOMPUTE)
        return inval("layer granularity needs every layer input X kept or offloaded");

  int rc = build_order(c, p);
  if (rc) return rc;

  // sizes
  const uint64_t T = p.T, h = p.h, f = p.f, es = p.esize;
  p.tbytes[TPS_T_X] = p.tbytes[TPS_T_A] = p.tbytes[TPS_T_O] = T * h * es;
  p.tbytes[TPS_T_X1] = p.tbytes[TPS_T_C] = T * h * es;
  p.tbytes[TPS_T_QKV] = T * (uint64_t)p.qw * es;
  p.tbytes[TPS_T_U] = T * (uint64_t)p.uw * es;
  p.tbytes[TPS_T_G] = T * f * es;
  p.tbytes[TPS_T_LSE] = (uint64_t)p.b * p.nh * p.s * 4;
  p.tbytes[TPS_T_LN1] = p.tbytes[TPS_T_LN2] = (p.llama ? 1 : 2) * T * 4;
  {
    uint64_t elems[TPS_P_COUNT];
    for (int i = 0; i < TPS_P_COUNT; ++i) elems[i] = (uint64_t)(p.prow[i] * p.pcol[i]);
    uint64_t po = 0, go = 0;
    for (int i = 0; i < TPS_P_COUNT; ++i) {
      p.poff[i] = po; po = align256(po + elems[i] * es);
      p.goff[i] = go; go = align256(go + elems[i] * 4);
    }
    p.pbytes = po; p.gbytes = go;
    // quantized block: matrices as one byte per element, their f32 row
    // scales after the vectors
    const bool is_mat[TPS_P_COUNT] = {true, false, true, false, true, false, true, false, false, false, false, false};
    const uint64_t rows[4] = {(uint64_t)p.prow[TPS_P_W_QKV], (uint64_t)p.prow[TPS_P_W_O],
                              (uint64_t)p.prow[TPS_P_W_1], (uint64_t)p.prow[TPS_P_W_2]};
    uint64_t qo = 0;
    for (int i = 0; i < TPS_P_COUNT; ++i) {
      p.qoff[i] = qo;
      qo = align256(qo + elems[i] * (is_mat[i] ? 1 : es));
    }
    for (int k = 0; k < 4; ++k) {
      p.qsoff[k] = qo;
      qo = align256(qo + rows[k] * 4);
    }
    p.qbytes = qo;
    p.hpbytes = p.quant == TPS_Q_FP8_ROW ? p.qbytes : p.pbytes;
  }

  // layouts: checkpoint slot, host slot, replay buffer
  p.kslot_off.assign((size_t)p.L * TPS_T_COUNT, kNone);
  p.oslot_off.assign((size_t)p.L * TPS_T_COUNT, kNone);
  p.replay_off.assign((size_t)p.L * TPS_T_COUNT, kNone);
  uint64_t so = 0, ho = 0, ro = 0;
  uint64_t shared_ro[TPS_T_COUNT];
  for (int t = 0; t < TPS_T_COUNT; ++t) shared_ro[t] = kNone;
  for (int l = 0; l < p.L; ++l) {
    for (int t = 0; t < TPS_T_COUNT; ++t) {
      const int pol = p.pol(l, t);
      const size_t k = (size_t)l * TPS_T_COUNT + t;
      if (pol == TPS_KEEP) { p.kslot_off[k] = so; so += align256(p.tbytes[t]); }
      if (pol == TPS_OFFLOAD) { p.oslot_off[k] = ho; ho += align256(p.tbytes[t]); }
      if (pol == TPS_RECOMPUTE) {
        if (p.granularity == TPS_GRAN_SEGMENT) {
          p.replay_off[k] = ro; ro += align256(p.tbytes[t]);
        } else {
          if (shared_ro[t] == kNone) { shared_ro[t] = ro; ro += align256(p.tbytes[t]); }
          p.replay_off[k] = shared_ro[t];
        }
      }
    }
  }
  p.kslot_bytes = so; p.oslot_bytes = ho; p.replay_bytes = ro;
  build_replay(p);

  // flops
  double unit_fwd = 0;
  for (int op = 0; op < OP_COUNT; ++op) unit_fwd += op_flops(p, op);
  p.fwd_flops = unit_fwd * p.L * p.M;
  p.bwd_flops = 2.0 * p.fwd_flops;
  double replay_mb = 0;
  for (int l = 0; l < p.L; ++l)
    for (int op = 0; op < OP_COUNT; ++op)
      if (p.replay_ops[l] & (1u << op)) replay_mb += op_flops(p, op);
  p.recompute_flops = replay_mb * p.M;

  // timing model of the order (compute and host-link rates from the hints):
  // forward and backward of one micro-batch, one micro-batch's offload copy
  const double rate = (c->tflops_hint > 0 ? c->tflops_hint : 1000.0) * 1e12;
  const double link = (c->link_gbps_hint > 0 ? c->link_gbps_hint : 50.0) * 1e9;
  const double tF = unit_fwd * p.L / rate;
  const double tB = (2.0 * unit_fwd * p.L + replay_mb) / rate;
  const double tc = (double)p.oslot_bytes / link;

  // offload victims
  if (c->offload_auto) {
    p.offload_mask = 0;
    if (p.oslot_bytes > 0) {
      std::vector<char> none(p.M, 0), chosen(p.M, 0);
      const double base = simulate_offload(p, none, tF, tB, tc);
      // slack between the end of F(mb) and the start of B(mb) without copies
      std::vector<double> slack(p.M, 0), t_end(p.op_kind.size(), 0);
      double t = 0;
      for (size_t i = 0; i < p.op_kind.size(); ++i) {
        t += p.op_kind[i] == TPS_OP_F ? tF : tB;
        t_end[i] = t;
      }
      for (int mb = 0; mb < p.M; ++mb) {
        const double b_start = t_end[p.pos_b[mb]] - tB;
        slack[mb] = b_start - t_end[p.pos_f[mb]];
      }
      std::vector<int> cand(p.M);
      std::iota(cand.begin(), cand.end(), 0);
      std::stable_sort(cand.begin(), cand.end(), [&](int a, int b2) { return slack[a] > slack[b2]; });
      // a victim is taken if the round keeps its time and the staging peak
      // drops (a micro-batch whose copies do not keep it off the device over
      // the peak would only add link traffic)
      int peak = assign_slots(p, tF, tB, tc);
      for (int mb : cand) {
        chosen[mb] = 1;
        if (simulate_offload(p, chosen, tF, tB, tc) <= base * 1.01) {
          p.offload_mask |= 1ull << mb;
          const int n = assign_slots(p, tF, tB, tc);
          if (n < peak) {
            peak = n;
            continue;
          }
          p.offload_mask &= ~(1ull << mb);
        }
        chosen[mb] = 0;
      }
    }
  } else {
    p.offload_mask = c->offload_mb_mask;
    if (p.M < 64 && (p.offload_mask >> p.M)) return inval("offload_mb_mask has bits beyond n_micro");
  }
  if (p.oslot_bytes == 0) p.offload_mask = 0;

  // slot and host-slot assignment over the order
  assign_slots(p, tF, tB, tc);

  // backward working buffers
  const uint64_t hb = align256(T * h * es), fb = align256(T * (uint64_t)p.uw * es),
                 qb = align256(T * (uint64_t)p.qw * es);
  p.defer_join = p.weights == TPS_W_RESIDENT && (p.granularity == TPS_GRAN_SEGMENT || p.n_replay_layers == 0);
  p.replay_independent = true;
  for (int l = 1; l < p.L; ++l)
    if (p.policy[(size_t)l * TPS_T_COUNT + TPS_T_X] == TPS_RECOMPUTE) p.replay_independent = false;
  {
    uint64_t o = 0;
    auto take = [&](uint64_t bytes) {
      const uint64_t r = o;
      o += bytes;
      return r;
    };
    const int ng = p.defer_join ? 3 : 2, sets = p.defer_join ? 2 : 1;
    for (int i = 0; i < 3; ++i) p.work.g[i] = i < ng ? take(hb) : p.work.g[0];
    for (int k = 0; k < 2; ++k) {
      p.work.dx1[k] = k < sets ? take(hb) : p.work.dx1[0];
      p.work.du[k] = k < sets ? take(fb) : p.work.du[0];
      p.work.dqkv[k] = k < sets ? take(qb) : p.work.dqkv[0];
    }
    p.work.t1 = take(hb);
    p.work.dvec = take(align256((uint64_t)p.b * p.nh * p.s * 4));
    p.work.dg = p.work.kvws = p.work.rope = p.work.zbias = kNone;
    if (p.llama) {
      p.work.dg = take(align256(T * f * es));
      if (p.nkv != p.nh) p.work.kvws = take(align256(T * 2 * h * es));
      p.work.rope = take(align256((uint64_t)p.s * p.d * 4));
      p.work.zbias = take(align256(h * es));
    }
    p.grp_n = 0;
    // (the slots of an operand must be consecutive rows: each slot a whole
    // number of 256-byte units)
    const bool rows_pack = (T * h * es) % 256 == 0 && (T * f * es) % 256 == 0 &&
                           (T * (uint64_t)p.uw * es) % 256 == 0 && (T * (uint64_t)p.qw * es) % 256 == 0;
    if (c->group_wgrad && p.granularity == TPS_GRAN_LAYER && p.M > 1 && rows_pack) {
      const uint64_t n = (uint64_t)p.M;
      p.grp_n = p.M;
      const uint64_t w_act[4] = {h, h, h, f};   // a, o, c, g
      for (int k = 0; k < 4; ++k) p.work.grp_act[k] = take(n * align256(T * w_act[k] * es));
      p.work.grp_du = take(n * fb);
      p.work.grp_dx1 = take(n * hb);
      p.work.grp_dqkv = take(n * qb);
      for (int k = 0; k < 2; ++k) p.work.grp_y[k] = take(n * hb);
    }
    p.work_bytes = o;
  }

  {
    const int64_t H = (int64_t)h, F = (int64_t)f;
    const int64_t gpt[Plan::BP_COUNT] = {3 * H, H, F, H, H, H, H, H};
    const int64_t lla[Plan::BP_COUNT] = {0, 0, 0, 0, 0, H, 0, H};
    const int64_t* widths = p.llama ? lla : gpt;
    p.bpc[0] = 0;
    for (int i = 0; i < Plan::BP_COUNT; ++i) p.bpc[i + 1] = p.bpc[i] + widths[i];
    p.bpart_segs = (int)colsum_segments(T);
    p.bpart_bytes = align256((uint64_t)p.bpart_segs * p.bpc[Plan::BP_COUNT] * 4);
  }

  // streamed window entry: parameter block, f32 gradient block, and with a
  // quantized reload the staging area its codes land in
  p.wwin_bytes = p.weights == TPS_W_STREAM
                     ? (uint64_t)p.window * (p.pbytes + p.gbytes + (p.quant ? align256(p.qbytes) : 0))
                     : 0;
  {
    const uint64_t mats[4] = {(uint64_t)p.qw * h, h * h, (uint64_t)p.uw * h, h * f};
    uint64_t o = 0;
    for (int i = 0; i < 4; ++i) {
      p.wtoff[i] = o;
      o = align256(o + mats[i] * es);
    }
    p.wt_bytes = o;
    p.wt_region = (p.weights == TPS_W_STREAM ? (uint64_t)p.window : (uint64_t)p.L) * p.wt_bytes;
  }

  p.off_kslots = 0;
  p.off_oslots = align256((uint64_t)p.n_kslots * p.kslot_bytes);
  p.off_replay = p.off_oslots + align256((uint64_t)p.n_oslots * p.oslot_bytes);
  p.off_work = p.off_replay + align256(p.replay_bytes);
  p.off_wwin = p.off_work + align256(p.work_bytes);
  p.off_bpart = p.off_wwin + align256(p.wwin_bytes);
  p.off_wt = p.off_bpart + (uint64_t)p.L * p.bpart_bytes;
  p.arena_bytes = p.off_wt + p.wt_region;
  p.host_bytes = (uint64_t)p.n_host_slots * p.oslot_bytes;

  int n_off = 0;
  for (int mb = 0; mb < p.M; ++mb) n_off += (p.offload_mask >> mb) & 1ull;
  p.h2d_bytes = (uint64_t)n_off * p.oslot_bytes;
  p.d2h_bytes = (uint64_t)n_off * p.oslot_bytes;
  if (p.weights == TPS_W_STREAM) {
    p.h2d_bytes += 2ull * p.L * p.hpbytes;
    p.d2h_bytes += (uint64_t)p.L * p.gbytes;
  }
  uint64_t per_mb_all = 0;
  for (int t = 0; t < TPS_T_COUNT; ++t) per_mb_all += align256(p.tbytes[t]);
  p.keep_all_bytes = (uint64_t)p.max_inflight * p.L * per_mb_all;
  p.predicted_peak = p.arena_bytes + (p.weights == TPS_W_RESIDENT ? (uint64_t)p.L * (p.pbytes + p.gbytes) : 0);

  *out = std::move(p);
  return TPS_OK;
}

void fill_plan_info(const Plan& p, tps_plan_info* info) {
  *info = tps_plan_info{};
  info->device_arena_bytes = p.arena_bytes;
  info->host_arena_bytes = p.host_bytes;
  info->slot_bytes = p.kslot_bytes;
  info->n_slots = p.n_kslots;
  info->offload_slot_bytes = p.oslot_bytes;
  info->n_offload_slots = p.n_oslots;
  info->n_host_slots = p.n_host_slots;
  info->max_inflight = p.max_inflight;
  info->replay_bytes = p.replay_bytes;
  info->work_bytes = p.work_bytes;
  info->weight_window_bytes = p.wwin_bytes;
  info->param_bytes = p.pbytes;
  info->grad_bytes = p.gbytes;
  info->keep_all_bytes = p.keep_all_bytes;
  info->predicted_peak_bytes = p.predicted_peak;
  info->offload_mb_mask = p.offload_mask;
  int n = 0;
  for (int mb = 0; mb < p.M; ++mb) n += (p.offload_mask >> mb) & 1ull;
  info->n_offload_mbs = n;
  info->n_replay_layers = p.n_replay_layers;
  info->fwd_flops = p.fwd_flops;
  info->bwd_flops = p.bwd_flops;
  info->recompute_flops = p.recompute_flops;
  info->h2d_bytes = p.h2d_bytes;
  info->d2h_bytes = p.d2h_bytes;
  info->wgrad_inline = p.wgrad_inline ? 1 : 0;
  info->group_wgrad_slots = p.grp_n;
}

}  // namespace tps

extern "C" int tps_plan(const tps_config* cfg, tps_plan_info* out) {
  tps::clear_error();
  if (!out) return tps::set_error(TPS_EINVAL, "tps_plan: null output");
  tps::Plan p;
  const int rc = tps::make_plan(cfg, &p);
  if (rc) return rc;
  tps::fill_plan_info(p, out);
  return TPS_OK;
}

extern "C" int tps_param_layout_q(const tps_config* cfg, uint64_t offsets[TPS_P_COUNT], uint64_t scale_offsets[4],
                                  uint64_t* bytes) {
  tps::clear_error();
  tps::Plan p;
  const int rc = tps::make_plan(cfg, &p);
  if (rc) return rc;
  for (int i = 0; i < TPS_P_COUNT; ++i)
    if (offsets) offsets[i] = p.qoff[i];
  for (int k = 0; k < 4; ++k)
    if (scale_offsets) scale_offsets[k] = p.qsoff[k];
  if (bytes) *bytes = p.qbytes;
  return TPS_OK;
}

extern "C" int tps_param_layout(const tps_config* cfg, uint64_t param_offsets[TPS_P_COUNT],
                                uint64_t* param_bytes, uint64_t grad_offsets[TPS_P_COUNT],
                                uint64_t* grad_bytes) {
  tps::clear_error();
  tps::Plan p;
  const int rc = tps::make_plan(cfg, &p);
  if (rc) return rc;
  for (int i = 0; i < TPS_P_COUNT; ++i) {
    if (param_offsets) param_offsets[i] = p.poff[i];
    if (grad_offsets) grad_offsets[i] = p.goff[i];
  }
  if (param_bytes) *param_bytes = p.pbytes;
  if (grad_bytes) *grad_bytes = p.gbytes;
  return TPS_OK;
}
