// T-Pipe two-chunk pipeline schedule and its unit-time simulator (host only).
//
// The model (paper, Section 4.1 "T-Pipe Schedule" and the appendix
// "Theoretical Analysis of T-Pipe"): p stages, each holding two chunks of
// layers, chunk 1 (shallow, layer block s) and chunk 2 (deep, layer block
// p + s).  A micro-batch's forward runs chunk 1 through stages 0..p-1, then
// chunk 2 through stages 0..p-1; its backward runs chunk 2 from stage p-1
// down to 0, then chunk 1 from p-1 down to 0.  Time is counted in T_unit,
// the forward of one chunk on one stage: a chunk forward takes 1, a chunk
// backward 2 (backward = twice the forward), and with block-wise T-Recomp
// (Section 4.2, "Addressing the Concerns") chunk 1 is recomputed as a task
// of its own (1 unit) that runs before that chunk's backward on the stage.
//
// Per-stage order.  Each stage repeats the pattern F(chunk 1), B(chunk 2),
// F(chunk 2), B(chunk 1) with one micro-batch per round of 6 units.  Chunk 1
// forwards pass the stages one unit apart, so F(chunk 1) of micro-batch j is
// at 6j + s on stage s; chunk 2's forward of j waits for the first pattern
// slot 3 units after a chunk-1 slot that follows the end of its chunk-1 pass,
// ceil((p-3)/6) rounds later (the forward interval of the appendix); the
// backward slots sit 2 units further back on each stage towards stage 0, so
// chunk 2's forward and backward round trip runs without waiting; chunk 1's
// backward follows ceil((2p-3)/6) rounds after chunk 2's on stage p-1 (the
// backward interval).  These slot times order each stage's tasks; with
// T-Recomp the recompute of (chunk 1, j) sits just before its backward, and
// chunk 2's tasks move `delay` rounds later in the order (the delay rounds of
// the appendix "Formalization on Delay Rounds at T-Recomp").  The simulator
// then starts every task as early as its stage and its dependencies allow
// (one task at a time per stage, in that order), which compresses the
// warm-up and cool-down.
//
// Activation accounting at a stage follows the appendix: the activations of
// (chunk, micro-batch) occupy one block from the start of its forward to the
// start of its backward on that stage; a recomputed chunk keeps none, and
// its regenerated activations occupy one buffer block from the start of the
// recompute to the end of the backward.
#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "errors.h"
#include "../../include/tpstage.h"

namespace {

int ceil_div(int a, int b) {  // b > 0, a of any sign
  return a >= 0 ? (a + b - 1) / b : -((-a) / b);
}

enum { K_F = TPS_OP_F, K_B = TPS_OP_B, K_R = TPS_OP_R };

struct Task {
  int kind, chunk, mb, stage;
  long key;        // order key on its stage (twice the slot time, recompute one less than its backward)
  int start = -1, end = -1;
};

struct Sim {
  int p, m, recomp, delay;
  int du[3];       // durations: forward, backward, recompute
  std::vector<Task> tasks;                 // all tasks
  std::vector<std::vector<int>> order;     // per stage: task indices in execution order
  int idx(int kind, int chunk, int mb, int stage) const {
    // layout: [mb][stage][slot], slot = F1, F2, B2, B1, R1
    const int slot = kind == K_F ? chunk - 1 : kind == K_B ? (chunk == 2 ? 2 : 3) : 4;
    return ((mb * p) + stage) * 5 + slot;
  }
};

void build(Sim& S) {
  const int p = S.p, m = S.m;
  const int kf = ceil_div(p - 3, 6), kb = ceil_div(2 * p - 3, 6);
  S.tasks.assign((size_t)m * p * 5, Task{});
  for (int j = 0; j < m; ++j) {
    const long r2 = (long)(j + kf + S.delay);   // chunk-2 round of micro-batch j
    const long b2_last = 6 * r2 + 3L * p + 1 - 2L * (p - 1);
    for (int s = 0; s < p; ++s) {
      const long f1 = 6L * j + s;
      const long f2 = 6 * r2 + 3 + s;
      const long b2 = 6 * r2 + 3L * p + 1 - 2L * s;
      const long b1 = b2_last + 3 + 6L * kb + 2L * (p - 1 - s);
      S.tasks[S.idx(K_F, 1, j, s)] = Task{K_F, 1, j, s, 2 * f1};
      S.tasks[S.idx(K_F, 2, j, s)] = Task{K_F, 2, j, s, 2 * f2};
      S.tasks[S.idx(K_B, 2, j, s)] = Task{K_B, 2, j, s, 2 * b2};
      S.tasks[S.idx(K_B, 1, j, s)] = Task{K_B, 1, j, s, 2 * b1};
      S.tasks[S.idx(K_R, 1, j, s)] = Task{K_R, 1, j, s, 2 * b1 - 1};
    }
  }
  S.order.assign(p, {});
  for (size_t i = 0; i < S.tasks.size(); ++i) {
    const Task& t = S.tasks[i];
    if (t.kind == K_R && !S.recomp) continue;
    S.order[t.stage].push_back((int)i);
  }
  for (auto& o : S.order)
    std::sort(o.begin(), o.end(), [&](int a, int b) {
      const Task &x = S.tasks[a], &y = S.tasks[b];
      if (x.key != y.key) return x.key < y.key;
      return a < b;
    });
}

// Tasks that must finish before t starts (besides the previous task of its stage).
int deps(const Sim& S, const Task& t, int out[2]) {
  const int p = S.p;
  int n = 0;
  if (t.kind == K_F) {
    if (t.stage > 0) out[n++] = S.idx(K_F, t.chunk, t.mb, t.stage - 1);
    else if (t.chunk == 2) out[n++] = S.idx(K_F, 1, t.mb, p - 1);
  } else if (t.kind == K_B) {
    if (t.stage < p - 1) out[n++] = S.idx(K_B, t.chunk, t.mb, t.stage + 1);
    else if (t.chunk == 2) out[n++] = S.idx(K_F, 2, t.mb, p - 1);
    else out[n++] = S.idx(K_B, 2, t.mb, 0);
    if (t.chunk == 1 && S.recomp) out[n++] = S.idx(K_R, 1, t.mb, t.stage);
  } else {
    out[n++] = S.idx(K_F, 1, t.mb, t.stage);
  }
  return n;
}

// As-soon-as-possible simulation in the per-stage orders; false on a
// dependency cycle (an order that waits for a later task of its own stage).
bool simulate(Sim& S) {
  const int p = S.p;
  std::vector<size_t> pos(p, 0);
  std::vector<int> free_at(p, 0);
  size_t left = 0;
  for (auto& o : S.order) left += o.size();
  for (auto& t : S.tasks) t.start = t.end = -1;
  while (left) {
    bool progressed = false;
    for (int s = 0; s < p; ++s) {
      while (pos[s] < S.order[s].size()) {
        Task& t = S.tasks[S.order[s][pos[s]]];
        int d[2];
        const int nd = deps(S, t, d);
        int ready = free_at[s];
        bool ok = true;
        for (int i = 0; i < nd; ++i) {
          const Task& u = S.tasks[d[i]];
          if (u.end < 0) { ok = false; break; }
          ready = std::max(ready, u.end);
        }
        if (!ok) break;
        t.start = ready;
        t.end = ready + S.du[t.kind];
        free_at[s] = t.end;
        ++pos[s];
        --left;
        progressed = true;
      }
    }
    if (!progressed) return false;
  }
  return true;
}

int makespan(const Sim& S) {
  int mk = 0;
  for (auto& t : S.tasks)
    if (t.end > mk) mk = t.end;
  return mk;
}

struct Blocks {
  int peak[2] = {0, 0}, peak_buf = 0, peak_total = 0;
};

// Peak activation blocks on stage s (see the accounting note at the top).
Blocks stage_blocks(const Sim& S, int s) {
  struct Ev {
    int t, d, what;   // what: 0 chunk 1, 1 chunk 2, 2 recompute buffer
  };
  std::vector<Ev> ev;
  for (int j = 0; j < S.m; ++j) {
    for (int c = 1; c <= 2; ++c) {
      if (c == 1 && S.recomp) continue;
      ev.push_back({S.tasks[S.idx(K_F, c, j, s)].start, +1, c - 1});
      ev.push_back({S.tasks[S.idx(K_B, c, j, s)].start, -1, c - 1});
    }
    if (S.recomp) {
      ev.push_back({S.tasks[S.idx(K_R, 1, j, s)].start, +1, 2});
      ev.push_back({S.tasks[S.idx(K_B, 1, j, s)].end, -1, 2});
    }
  }
  // releases before acquisitions at the same instant
  std::sort(ev.begin(), ev.end(), [](const Ev& a, const Ev& b) { return a.t != b.t ? a.t < b.t : a.d < b.d; });
  Blocks B;
  int cur[3] = {0, 0, 0}, tot = 0;
  for (auto& e : ev) {
    cur[e.what] += e.d;
    tot += e.d;
    if (e.what < 2) B.peak[e.what] = std::max(B.peak[e.what], cur[e.what]);
    else B.peak_buf = std::max(B.peak_buf, cur[2]);
    B.peak_total = std::max(B.peak_total, tot);
  }
  return B;
}

// Idle time of stage s inside [a, b): the interval less the tasks of the
// stage that run in it (tasks of one stage never overlap).
int stage_idle(const Sim& S, int s, int a, int b) {
  if (b <= a) return 0;
  int busy = 0;
  for (int i : S.order[s]) {
    const Task& t = S.tasks[i];
    busy += std::max(0, std::min(t.end, b) - std::max(t.start, a));
  }
  return (b - a) - busy;
}

// The two host-transfer windows of the appendix "Scalability of T-Offload"
// on stage s.  Offload: idle time from the end of chunk 2's last backward to
// the start of chunk 1's last backward (the cool-down gap that holds the
// gradient offload and host optimizer step of chunk 2).  Upload: idle time
// from the stage's first task to chunk 2's first forward (the warm-up gap
// that holds the reload of chunk 2's weights).
void stage_windows(const Sim& S, int s, int* offload, int* upload) {
  int b2_end = 0, b1_start = 0, first = -1, f2_start = -1;
  for (int i : S.order[s]) {
    const Task& t = S.tasks[i];
    if (t.kind == K_B && t.chunk == 2) b2_end = std::max(b2_end, t.end);
    if (t.kind == K_B && t.chunk == 1) b1_start = std::max(b1_start, t.start);
    if (first < 0 || t.start < first) first = t.start;
    if (t.kind == K_F && t.chunk == 2 && (f2_start < 0 || t.start < f2_start)) f2_start = t.start;
  }
  *offload = stage_idle(S, s, b2_end, b1_start);
  *upload = stage_idle(S, s, first, f2_start);
}

}  // namespace

extern "C" int tps_tpipe_schedule(const tps_tpipe_config* cfg, int32_t stage, tps_tpipe_task* tasks,
                                  int32_t max_tasks, int32_t* n_tasks, tps_tpipe_result* out) {
  tps::clear_error();
  if (!cfg || !out) return tps::set_error(TPS_EINVAL, "tps_tpipe_schedule: null argument");
  const int p = cfg->stages, m = cfg->micro;
  if (p < 1 || p > 256 || m < 1 || m > 4096) return tps::set_error(TPS_EINVAL, "tps_tpipe_schedule: stages in 1..256, micro in 1..4096");
  if (stage < 0 || stage >= p) return tps::set_error(TPS_EINVAL, "tps_tpipe_schedule: stage out of range");
  if (cfg->delay < -1 || cfg->delay > 64) return tps::set_error(TPS_EINVAL, "tps_tpipe_schedule: delay in -1..64");
  if (max_tasks > 0 && !tasks) return tps::set_error(TPS_EINVAL, "tps_tpipe_schedule: null task buffer");
  Sim S;
  S.p = p;
  S.m = m;
  S.recomp = cfg->t_recomp ? 1 : 0;
  S.du[K_F] = 1;
  S.du[K_B] = 2;
  S.du[K_R] = 1;
  // the delay: given, or the smallest number of rounds that reaches the
  // shortest makespan (a delay too small makes chunk-2 forwards collide with
  // the recompute-lengthened rounds and wait; more rounds than needed only
  // hold activations longer)
  int best_k = cfg->delay, best_mk = -1;
  if (cfg->delay < 0) {
    const int kmax = 8;
    for (int k = 0; k <= kmax; ++k) {
      S.delay = k;
      build(S);
      if (!simulate(S)) continue;
      const int mk = makespan(S);
      if (best_mk < 0 || mk < best_mk) {
        best_mk = mk;
        best_k = k;
      }
    }
    if (best_mk < 0) return tps::set_error(TPS_EINVAL, "tps_tpipe_schedule: no feasible delay");
  }
  S.delay = best_k;
  build(S);
  if (!simulate(S)) return tps::set_error(TPS_EINVAL, "tps_tpipe_schedule: the per-stage order deadlocks for this delay");

  memset(out, 0, sizeof(*out));
  out->delay = S.delay;
  out->makespan = makespan(S);
  out->busy = m * (2 * S.du[K_F] + 2 * S.du[K_B] + (S.recomp ? S.du[K_R] : 0));
  out->bubble_ratio = out->makespan > 0 ? (double)(out->makespan - out->busy) / out->makespan : 0.0;
  const Blocks b = stage_blocks(S, stage);
  out->peak_blocks_chunk1 = b.peak[0];
  out->peak_blocks_chunk2 = b.peak[1];
  out->peak_buffer_blocks = b.peak_buf;
  out->peak_blocks = b.peak_total;
  for (int s = 0; s < p; ++s) out->max_stage_peak_blocks = std::max(out->max_stage_peak_blocks, stage_blocks(S, s).peak_total);
  // lifespans of the middle micro-batch (steady state for m >= 2p)
  const int jm = m / 2;
  out->life_chunk1 = S.tasks[S.idx(K_B, 1, jm, stage)].start - S.tasks[S.idx(K_F, 1, jm, stage)].start;
  out->life_chunk2 = S.tasks[S.idx(K_B, 2, jm, stage)].start - S.tasks[S.idx(K_F, 2, jm, stage)].start;
  stage_windows(S, stage, &out->offload_window, &out->upload_window);

  const auto& ord = S.order[stage];
  if (n_tasks) *n_tasks = (int32_t)ord.size();
  for (size_t i = 0; i < ord.size() && (int32_t)i < max_tasks; ++i) {
    const Task& t = S.tasks[ord[i]];
    tasks[i].kind = t.kind;
    tasks[i].chunk = t.chunk;
    tasks[i].mb = t.mb;
    tasks[i].start = t.start;
    tasks[i].end = t.end;
  }
  return TPS_OK;
}
