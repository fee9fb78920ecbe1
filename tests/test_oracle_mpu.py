"""Pins of the MPU planner reference (CPU only).

* the budget ladder of Eq. 6 against ladders worked out by hand;
* the worked example of Pipeline Scheduling: 2M tokens on four stages give two waves at budget M
  and four at M/2, and the planner picks M/2;
* Eq. 7: pieces larger than half a budget cannot share a wave, so they count as waves on their own;
* hand-built cases for the 12.5 % rule, the hysteresis, the fragment floor, the lone-wave wait
  and partial acceptance;
* invariants over seeded traces: budgets, lanes, FCFS order, and every prompt tiled exactly once.
"""
import numpy as np
import pytest

from oracle import mpu as om


def test_ladder_by_hand():
    assert om.budget_ladder(16384, 512, 64) == [16384, 8192, 4096, 2048, 1024, 512]
    assert om.budget_ladder(16384, 8192, 64) == [16384, 8192]
    # 65 blocks: half is 2080, aligned down to 2048
    assert om.budget_ladder(4160, 1024, 64) == [4160, 2048, 1024]
    # the floor stops the halving even when half of a step is below it
    assert om.budget_ladder(3072, 1024, 512) == [3072, 1536, 1024]
    assert om.budget_ladder(512, 512, 64) == [512]
    for bad in [(16384, 100, 64), (16384, 32768, 64), (16032, 512, 64), (16384, 32, 64)]:
        with pytest.raises(ValueError):
            om.budget_ladder(*bad)


def run_trace(pl, requests, admission=()):
    """Admit everything, then plan / commit until done, retiring the oldest wave when the ring is full.
    Returns the list of waves (each a list of spans) and the budgets used."""
    for rid, s, e in requests:
        pl.admit(rid, s, e)
    waves, budgets = [], []
    for _ in range(10000):
        spans, b = pl.plan(admission_pending=False)
        if not spans:
            if pl.ring:
                pl.retire()
                continue
            break
        pl.commit(spans)
        waves.append(spans)
        budgets.append(b)
    return waves, budgets


def test_worked_example_two_m_tokens_on_four_stages():
    M = 16384
    reqs = [(i, 0, 4096) for i in range(8)]          # 2M tokens in total
    mpu = om.Planner(max_budget=M, min_budget=M // 2, block=64, stages=4, fills=2, max_lanes=64)
    waves, budgets = run_trace(mpu, reqs)
    assert budgets[0] == M // 2 and len(waves) == 4
    greedy = om.Planner(max_budget=M, min_budget=M, block=64, stages=4, fills=2, max_lanes=64)
    waves_g, budgets_g = run_trace(greedy, reqs)
    assert set(budgets_g) == {M} and len(waves_g) == 2


def test_pieces_above_half_a_budget_count_as_waves():
    # three pieces of 0.6 M: W / M = 1.8, but no two of them can share a wave
    assert om.waves_at_least(3 * 9830, [9830] * 3, 16384, 3)
    assert not om.waves_at_least(3 * 9830, [9830] * 3, 16384, 4)
    # pieces of exactly half a budget can share a wave
    assert not om.waves_at_least(3 * 8192, [8192] * 3, 16384, 3)


def test_thinning_limited_by_newly_split_share():
    ladder = om.budget_ladder(16384, 2048, 64)
    S, R = 12, 8
    # ten pieces of 15000: at 16384 about 9.2 waves (>= R, < S); halving would split all of them
    assert om.choose_budget(ladder, 150000, [15000] * 10, S, R, 125) == 16384
    # the same tokens in pieces of 6000 are not split by halving: thinning continues to 8192
    assert om.choose_budget(ladder, 150000, [6000] * 25, S, R, 125) == 8192
    # with few waves (< R) thinning is not limited: the budget falls to where n(b) >= S
    assert om.choose_budget(ladder, 60000, [15000] * 4, S, R, 125) == 4096
    # nothing qualifies: the floor
    assert om.choose_budget(ladder, 1000, [1000], S, R, 125) == 2048


def test_budget_hysteresis():
    pl = om.Planner(max_budget=16384, min_budget=2048, block=64, stages=4, fills=2, max_lanes=64)
    R = pl.R
    pl.budget = 4096
    big_w, big_p = 10 ** 7, [1000]
    # one halving up (to 8192) is adopted only after R/2 decisions asking for it
    for i in range(R // 2 - 1):
        pl._update_budget(8192, big_w, big_p)
        assert pl.budget == 4096
    pl._update_budget(8192, big_w, big_p)
    assert pl.budget == 8192
    # two halvings up at once: immediately
    pl.budget = 2048
    pl._update_budget(8192, big_w, big_p)
    assert pl.budget == 8192
    # a decrease needs R decisions in a row and the current budget to be a full wave short
    small_w, small_p = 8192 * 3, [4096] * 6
    for i in range(R - 1):
        pl._update_budget(2048, small_w, small_p)
        assert pl.budget == 8192
    pl._update_budget(2048, small_w, small_p)
    assert pl.budget == 2048
    # ... and an interruption restarts the count
    pl.budget = 8192
    for i in range(R - 1):
        pl._update_budget(2048, small_w, small_p)
    pl._update_budget(8192, small_w, small_p)
    pl._update_budget(2048, small_w, small_p)
    assert pl.budget == 8192
    # the hysteresis check: enough work at the current budget blocks the decrease
    pl2 = om.Planner(max_budget=16384, min_budget=2048, block=64, stages=4, fills=2, max_lanes=64)
    pl2.budget = 8192
    for i in range(2 * R):
        pl2._update_budget(4096, 8192 * pl2.S, [100])
    assert pl2.budget == 8192


def test_fragment_floor_and_fcfs():
    M, bmin = 16384, 4096
    pl = om.Planner(max_budget=M, min_budget=bmin, block=64, stages=1, fills=1, max_lanes=8)
    pl.budget = M
    pl.admit(0, 0, 14000)     # leaves 2384 < max(b_min, b / 2) = 8192 of space
    pl.admit(1, 0, 20000)
    pl.admit(2, 0, 100)
    spans, b = pl.plan()
    # request 1 would be a 2384-token fragment: not placed, and request 2 does not overtake it
    assert b == M and spans == [(0, 0, 14000)]


def test_lone_small_wave_waits_once_for_admission():
    pl = om.Planner(max_budget=16384, min_budget=8192, block=64, stages=4, fills=1, max_lanes=8)
    pl.admit(0, 0, 30000)
    spans, b = pl.plan()
    pl.commit(spans)                              # the ring is now busy
    pl.admit(1, 0, 500)
    pl.queue[0].pos = pl.queue[0].end             # only the small request is left
    assert pl.plan(admission_pending=True)[0] == []
    assert pl.plan(admission_pending=True)[0] == [(1, 0, 500)]
    # without pending admission it is scheduled at once
    pl2 = om.Planner(max_budget=16384, min_budget=8192, block=64, stages=4, fills=1, max_lanes=8)
    pl2.admit(0, 0, 30000)
    pl2.commit(pl2.plan()[0])
    pl2.admit(1, 0, 500)
    pl2.queue[0].pos = pl2.queue[0].end
    assert pl2.plan(admission_pending=False)[0] == [(1, 0, 500)]


def test_partial_acceptance_advances_by_accepted_spans_only():
    pl = om.Planner(max_budget=16384, min_budget=8192, block=64, stages=4, fills=1, max_lanes=8)
    pl.admit(7, 100, 40000)
    spans, _ = pl.plan()
    assert spans[0][:2] == (7, 100)
    pl.commit([(7, 100, 3000)])
    spans, _ = pl.plan()
    assert spans[0][:2] == (7, 3100)
    with pytest.raises(ValueError):
        pl.commit([(7, 100, 10)])                 # not at the request's position


def test_inflight_chunks_keep_the_budget_up():
    """W counts the latest committed chunk of a request while its wave is in the ring."""
    pl = om.Planner(max_budget=16384, min_budget=4096, block=64, stages=2, fills=1, max_lanes=8)
    pl.admit(0, 0, 16384 * 4)
    spans, _ = pl.plan()
    pl.commit(spans)
    W, pieces = pl.work()
    assert W == 16384 * 4 and pieces == [16384 * 3, spans[0][2]]
    pl.retire()
    W2, _ = pl.work()
    assert W2 == 16384 * 3
    pl_no = om.Planner(max_budget=16384, min_budget=4096, block=64, stages=2, fills=1, max_lanes=8,
                       count_inflight=False)
    pl_no.admit(0, 0, 16384 * 4)
    pl_no.commit(pl_no.plan()[0])
    assert pl_no.work()[0] == 16384 * 3


@pytest.mark.parametrize("seed", range(6))
def test_trace_invariants(seed):
    rng = np.random.default_rng(seed)
    M, bmin, B = 16384, 2048, 64
    P, F, lanes = int(rng.integers(1, 9)), int(rng.integers(1, 3)), int(rng.integers(1, 17))
    pl = om.Planner(max_budget=M, min_budget=bmin, block=B, stages=P, fills=F, max_lanes=lanes)
    reqs = []
    for rid in range(int(rng.integers(1, 40))):
        s = int(rng.integers(0, 4)) * 64
        reqs.append((rid, s, s + int(rng.integers(1, 60000))))
    waves, budgets = run_trace(pl, reqs)
    covered = {rid: [] for rid, _, _ in reqs}
    for spans, b in zip(waves, budgets):
        assert b in pl.ladder
        assert 0 < sum(l for _, _, l in spans) <= b
        assert len(spans) <= lanes
        ids = [r for r, _, _ in spans]
        assert len(set(ids)) == len(ids)
        for rid, s, l in spans:
            covered[rid].append((s, l))
    for rid, s, e in reqs:
        pos = s
        for st, l in covered[rid]:
            assert st == pos
            pos += l
        assert pos == e
