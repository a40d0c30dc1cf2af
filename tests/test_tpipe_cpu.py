"""T-Pipe two-chunk schedule and unit-time simulator (tps_tpipe_schedule, host
only) pinned to the closed forms the paper derives for it:

* appendix "Theoretical Analysis of T-Pipe": total time 6(m + p - 1) T_unit,
  hence the bubble ratio (p - 1)/(m + p - 1); activation lifespans of chunk 2
  (3p - 2 T_unit, start of forward to start of backward) and chunk 1 (its
  forward, the forward interval (3 + 6 ceil((p-3)/6) - p), chunk 2's
  lifespan, the backward interval (3 + 6 ceil((2p-3)/6) - 2p) and its
  backward); peak blocks ceil(2/3 + ceil((p-3)/6) + ceil((2p-3)/6) + p/2) for
  chunk 1 and ceil((3p-2)/6) for chunk 2, about 75% of m_a together;
* appendix "Formalization on Delay Rounds at T-Recomp": the delay k is the
  smallest integer with T_fwd_interval - dT_fwd_interval + 7k >= 0;
* appendix "Theoretical Analysis of T-Recomp": chunk 2's lifespan
  3p + ceil((p-1)/2) - 2, one recompute buffer block, about 25% of m_a, and
  total time at most 6p + 7(m - 1) T_unit;
* appendix "Scalability of T-Offload": the cool-down window between the end
  of chunk 2's backward and chunk 1's last backward holds
  (p - ceil((2p-3)/6) - 1) chunk backwards (2 T_unit each), the warm-up
  window before chunk 2's first forward (p - ceil((p-3)/6) - 1) chunk
  forwards, growing as 2p/3 and 5p/6 for large p.

None of these formulas is used by the simulator: it only orders each
stage's tasks by the slot pattern and runs them as early as dependencies
allow."""

import math

import pytest

from paper_2503_03182_amd import tpstage as T


def cdiv(a, b):
    return -(-a // b)


def k_formula(p):
    """Delay rounds of the appendix's optimisation problem (p >= 3)."""
    t_fwd_interval = 3 + 6 * cdiv(p - 3, 6) - p
    d_interval = cdiv(p - 1, 2) - cdiv(p - 3, 6) - 1
    k = 0
    while t_fwd_interval - d_interval + 7 * k < 0:
        k += 1
    return k


@pytest.mark.parametrize("p", list(range(1, 41)))
def test_tpipe_total_time_and_bubble_ratio(p):
    for m in (1, 2, p, 2 * p, 3 * p + 1):
        r, tasks = T.tpipe_schedule(p, m)
        assert r["makespan"] == 6 * (m + p - 1), (p, m)
        assert r["busy"] == 6 * m
        assert r["bubble_ratio"] == pytest.approx((p - 1) / (m + p - 1))
        assert len(tasks) == 4 * m and r["delay"] == 0


@pytest.mark.parametrize("p", list(range(2, 41)))
def test_tpipe_peak_activation_and_lifespans(p):
    m = 4 * p
    r, _ = T.tpipe_schedule(p, m)
    c1 = math.ceil(2 / 3 + cdiv(p - 3, 6) + cdiv(2 * p - 3, 6) + p / 2)
    c2 = cdiv(3 * p - 2, 6)
    assert (r["peak_blocks_chunk1"], r["peak_blocks_chunk2"]) == (c1, c2)
    # the two chunks need not peak at the same instant
    assert max(c1, c2) <= r["peak_blocks"] <= c1 + c2
    assert r["peak_blocks"] <= r["max_stage_peak_blocks"]
    assert r["life_chunk2"] == 3 * p - 2                      # T_fwd_chunk2 + T_bwd_chunk2 - 2 T_unit
    f_int = 3 + 6 * cdiv(p - 3, 6) - p
    b_int = 3 + 6 * cdiv(2 * p - 3, 6) - 2 * p
    assert r["life_chunk1"] == p + f_int + (3 * p - 2) + b_int + 2 * p
    # blocks are m_a / 2p each: the peak tends to 75% of m_a
    assert 0.75 <= (c1 + c2) / (2 * p) <= 0.75 + 2.5 / p


def test_tpipe_steady_state_round_is_six_units():
    for p in (2, 5, 8, 13):
        a = T.tpipe_schedule(p, 3 * p)[0]["makespan"]
        b = T.tpipe_schedule(p, 3 * p + 1)[0]["makespan"]
        assert b - a == 6


def test_tpipe_figure_statement_stage0_p4():
    """With four stages, stage 0 starts chunk 2 of the fourth micro-batch
    before it releases chunk 2 of the third (the release is the start of that
    chunk's backward)."""
    _, tasks = T.tpipe_schedule(4, 8, stage=0)
    start = {(k, c, mb): s for k, c, mb, s, _ in tasks}
    assert start[("F", 2, 3)] < start[("B", 2, 2)]


@pytest.mark.parametrize("t_recomp", [False, True])
@pytest.mark.parametrize("p", [1, 2, 3, 4, 7, 8, 12])
def test_schedule_respects_dependencies_and_stage_exclusivity(p, t_recomp):
    """Every stage runs one task at a time; a chunk's forward follows the
    previous stage's (chunk 2 on stage 0 follows chunk 1 on stage p-1), a
    backward follows the next stage's (chunk 2 on stage p-1 follows its
    forward, chunk 1 on stage p-1 follows chunk 2 on stage 0), and a
    recompute precedes its backward; durations 1 / 2 / 1 T_unit."""
    m = 2 * p + 3
    lists = [T.tpipe_schedule(p, m, stage=s, t_recomp=t_recomp)[1] for s in range(p)]
    when = {}
    for s, tasks in enumerate(lists):
        prev_end = 0
        for k, c, mb, a, b in tasks:
            assert a >= prev_end
            assert b - a == {"F": 1, "B": 2, "R": 1}[k]
            prev_end = b
            when[(k, c, mb, s)] = (a, b)
    assert len(when) == p * m * (5 if t_recomp else 4)
    for (k, c, mb, s), (a, _) in when.items():
        if k == "F":
            dep = ("F", c, mb, s - 1) if s > 0 else (("F", 1, mb, p - 1) if c == 2 else None)
        elif k == "B":
            dep = ("B", c, mb, s + 1) if s < p - 1 else (("F", 2, mb, p - 1) if c == 2 else ("B", 2, mb, 0))
            if c == 1 and t_recomp:
                assert when[("R", 1, mb, s)][1] <= a
        else:
            dep = ("F", 1, mb, s)
        if dep is not None:
            assert when[dep][1] <= a, ((k, c, mb, s), dep)


@pytest.mark.parametrize("p", list(range(4, 41)))
def test_trecomp_delay_rounds_match_the_appendix(p):
    """The smallest delay that reaches the shortest simulated time equals the
    appendix's optimisation result for every p in 4..40 (k = 0, 1 or 2)."""
    r, _ = T.tpipe_schedule(p, 2 * p + 5, t_recomp=True)
    assert r["delay"] == k_formula(p)


def test_trecomp_delay_small_pipelines():
    """p = 3 is the one place the simulated delay (1) exceeds the appendix's
    formula (0): without it chunk 2 of stage 0 starts one unit late."""
    assert k_formula(3) == 0
    assert T.tpipe_schedule(3, 11, t_recomp=True)[0]["delay"] == 1
    assert T.tpipe_schedule(3, 11, t_recomp=True, delay=0)[0]["makespan"] == \
        T.tpipe_schedule(3, 11, t_recomp=True, delay=1)[0]["makespan"] + 1


@pytest.mark.parametrize("p", list(range(2, 41)))
def test_trecomp_lifespan_buffer_and_total_time(p):
    for m in (2 * p, 2 * p + 5):
        r, tasks = T.tpipe_schedule(p, m, t_recomp=True)
        assert len(tasks) == 5 * m
        assert r["life_chunk2"] == 3 * p + cdiv(p - 1, 2) - 2
        # blocks held by chunk 2: ceil(life / 7); the appendix writes floor(p/2),
        # which is the same number for even p (one more for odd p)
        assert r["peak_blocks_chunk2"] == cdiv(r["life_chunk2"], 7) == cdiv(p, 2)
        if p % 2 == 0:
            assert r["peak_blocks_chunk2"] == p // 2
        assert r["peak_blocks_chunk1"] == 0 and r["peak_buffer_blocks"] == 1
        # about 25% of m_a
        assert (r["peak_blocks"]) / (2 * p) <= 0.25 + 1.0 / p
        assert r["makespan"] <= 6 * p + 7 * (m - 1)
        assert r["busy"] == 7 * m


def test_trecomp_steady_state_round_is_seven_units():
    for p in (4, 8, 9, 16):
        a = T.tpipe_schedule(p, 3 * p, t_recomp=True)[0]["makespan"]
        b = T.tpipe_schedule(p, 3 * p + 1, t_recomp=True)[0]["makespan"]
        assert b - a == 7


def test_trecomp_needs_less_activation_than_tpipe():
    for p in (4, 8, 16):
        plain = T.tpipe_schedule(p, 4 * p)[0]["peak_blocks"]
        rec = T.tpipe_schedule(p, 4 * p, t_recomp=True)[0]["peak_blocks"]
        assert rec < plain / 2


def test_chunk_orders_split():
    _, tasks = T.tpipe_schedule(4, 6, stage=1, t_recomp=True)
    o1, o2, calls = T.chunk_orders(tasks)
    for o in (o1, o2):
        assert sorted(o) == sorted([("F", j) for j in range(6)] + [("B", j) for j in range(6)])
        for j in range(6):
            assert o.index(("F", j)) < o.index(("B", j))
    assert len(calls) == 24


def test_tpipe_argument_errors():
    for args in [(0, 4), (4, 0), (300, 4)]:
        with pytest.raises(T.TpsError) as e:
            T.tpipe_schedule(*args)
        assert e.value.code == T.TPS_EINVAL
    with pytest.raises(T.TpsError):
        T.tpipe_schedule(4, 4, stage=4)
    with pytest.raises(T.TpsError):
        T.tpipe_schedule(4, 4, delay=-2)


def idle_between(tasks, a, b):
    """Idle time of a stage's task list inside [a, b), counted from the
    simulated start and end times."""
    if b <= a:
        return 0
    busy = sum(max(0, min(e, b) - max(st, a)) for _, _, _, st, e in tasks)
    return (b - a) - busy


@pytest.mark.parametrize("p", list(range(1, 41)))
def test_t_offload_windows_match_the_appendix(p):
    """The windows equal the closed forms once the mini-batch has more
    micro-batches than chunk 1's backward lags chunk 2's (ceil((2p-3)/6)
    rounds) and chunk 2's forward lags chunk 1's (ceil((p-3)/6) rounds);
    shorter mini-batches leave larger windows.  The same on every stage."""
    lag_b, lag_f = cdiv(2 * p - 3, 6), cdiv(p - 3, 6)
    w_off = 2 * (p - lag_b - 1)          # chunk backwards of 2 T_unit
    w_up = p - lag_f - 1                 # chunk forwards of 1 T_unit
    stages = sorted({0, p // 2, p - 1})
    for m in list(range(1, lag_b + 3)) + [2 * p, 3 * p + 1]:
        for s in stages:
            r, _ = T.tpipe_schedule(p, m, stage=s)
            if m >= lag_b + 1:
                assert r["offload_window"] == w_off, (p, m, s)
            else:
                assert r["offload_window"] >= w_off, (p, m, s)
            if m >= lag_f + 1:
                assert r["upload_window"] == w_up, (p, m, s)
            else:
                assert r["upload_window"] >= w_up, (p, m, s)


@pytest.mark.parametrize("t_recomp", [False, True])
def test_t_offload_windows_recount_from_the_timeline(t_recomp):
    for p, m in [(1, 3), (3, 5), (4, 8), (7, 9), (8, 16), (13, 30)]:
        for s in sorted({0, p // 2, p - 1}):
            r, tasks = T.tpipe_schedule(p, m, stage=s, t_recomp=t_recomp)
            b2_end = max(e for k, c, _, _, e in tasks if k == "B" and c == 2)
            b1_start = max(st for k, c, _, st, _ in tasks if k == "B" and c == 1)
            first = min(st for _, _, _, st, _ in tasks)
            f2_start = min(st for k, c, _, st, _ in tasks if k == "F" and c == 2)
            assert r["offload_window"] == idle_between(tasks, b2_end, b1_start), (p, m, s)
            assert r["upload_window"] == idle_between(tasks, first, f2_start), (p, m, s)


def test_t_offload_windows_grow_linearly_with_stages():
    """Large-p forms of the two conditions: T_step / T_bwd * 3 / (2p) <= 1 and
    T_upload / T_fwd * 6 / (5p) <= 1, i.e. windows of about 2p/3 chunk
    backwards and 5p/6 chunk forwards."""
    for p in (24, 48, 96, 192):
        r, _ = T.tpipe_schedule(p, 2 * p)
        assert abs(r["offload_window"] / 2 - 2 * p / 3) <= 2
        assert abs(r["upload_window"] - 5 * p / 6) <= 2


def test_t_offload_stage_count():
    # windows in T_unit at m = 2p: offload 2 (p - ceil((2p-3)/6) - 1), upload p - ceil((p-3)/6) - 1
    def first(pred):
        return next(p for p in range(1, 257) if pred(p))

    for t_off, t_up, unit in [(0.0, 0.0, 1.0), (18.0, 3.8, 1.0), (1619.0, 345.0, 90.0), (7.0, 0.5, 0.25)]:
        p_off, p_up = T.tpipe_t_offload_stages(t_off, t_up, unit)
        assert p_off == first(lambda p: t_off <= 2 * (p - cdiv(2 * p - 3, 6) - 1) * unit)
        assert p_up == first(lambda p: t_up <= (p - cdiv(p - 3, 6) - 1) * unit)
    assert T.tpipe_t_offload_stages(18.0, 3.8, 1.0) == (15, 6)
    assert T.tpipe_t_offload_stages(1e9, 1.0, 1.0, max_stages=16) == (None, 2)
    for bad in [(1.0, 1.0, 0.0), (-1.0, 1.0, 1.0), (1.0, -1.0, 1.0)]:
        with pytest.raises(ValueError):
            T.tpipe_t_offload_stages(*bad)
