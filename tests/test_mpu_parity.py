"""The native MPU planner (C ABI) against the reference planner: identical decisions, decision by
decision, on seeded traces of admissions, plans, partial acceptances and retirements (CPU only)."""
import numpy as np
import pytest

import paper_2609_35263_amd as wp
from oracle import mpu as om


def test_ladder_matches():
    for M, bmin, B in [(16384, 512, 64), (16384, 8192, 64), (4160, 1024, 64), (3072, 1024, 512), (512, 512, 64)]:
        assert wp.mpu_budget_ladder(M, bmin, B) == om.budget_ladder(M, bmin, B)
    with pytest.raises(wp.WaveppError):
        wp.mpu_budget_ladder(16384, 100, 64)


def test_worked_example_native():
    M = 16384
    native = wp.MpuPlanner(max_budget=M, min_budget=M // 2, block=64, stages=4, fills=2, max_lanes=64)
    for i in range(8):
        native.admit(i, 0, 4096)
    waves = []
    while True:
        spans, b = native.plan()
        if not spans:
            break
        native.commit(spans)
        waves.append((b, spans))
    assert len(waves) == 4 and {b for b, _ in waves} == {M // 2}


def test_commit_rejects_position_mismatch():
    native = wp.MpuPlanner(max_budget=16384, min_budget=8192, block=64, stages=2, fills=1, max_lanes=4)
    native.admit(3, 64, 9000)
    with pytest.raises(wp.WaveppError) as e:
        native.commit([(3, 0, 100)])
    assert e.value.status == -5
    with pytest.raises(wp.WaveppError):
        native.commit([(4, 0, 100)])


CONFIGS = [
    dict(max_budget=16384, min_budget=8192, block=64, stages=4, fills=2, max_lanes=64),
    dict(max_budget=16384, min_budget=512, block=64, stages=8, fills=2, max_lanes=32),
    dict(max_budget=16384, min_budget=8192, block=64, stages=8, fills=1, max_lanes=256, count_inflight=False),
    dict(max_budget=8192, min_budget=1024, block=128, stages=2, fills=3, max_lanes=4, split_permille=0),
    dict(max_budget=4096, min_budget=256, block=64, stages=1, fills=1, max_lanes=2, split_permille=1000),
]


@pytest.mark.parametrize("cfg", range(len(CONFIGS)))
@pytest.mark.parametrize("seed", range(4))
def test_native_matches_reference_decision_by_decision(cfg, seed):
    c = CONFIGS[cfg]
    rng = np.random.default_rng(100 * cfg + seed)
    ref = om.Planner(**c)
    nat = wp.MpuPlanner(**c)
    next_id, steps = 0, 0
    for step in range(400):
        op = rng.random()
        if op < 0.25 or not ref.queue:
            start = int(rng.integers(0, 50)) * 64
            length = int(rng.choice([rng.integers(1, 2000), rng.integers(2000, 40000), rng.integers(40000, 200000)]))
            ref.admit(next_id, start, start + length)
            nat.admit(next_id, start, start + length)
            next_id += 1
        elif op < 0.85:
            pending = bool(rng.random() < 0.3)
            s_ref, b_ref = ref.plan(admission_pending=pending)
            s_nat, b_nat = nat.plan(admission_pending=pending)
            assert s_nat == [tuple(x) for x in s_ref], (step, s_nat, s_ref)
            if s_ref:
                assert b_nat == b_ref
                accepted = list(s_ref)
                if rng.random() < 0.2:                      # the scheduler accepts less
                    accepted = accepted[:max(1, len(accepted) - 1)]
                    rid, st, ln = accepted[-1]
                    accepted[-1] = (rid, st, max(1, int(ln * rng.uniform(0.3, 1.0))))
                assert nat.commit(accepted) == ref.commit(accepted)
                steps += 1
        elif ref.ring:
            ref.retire()
            nat.retire()
        st = nat.state()
        W, _ = ref.work()
        assert (st["work"], st["budget"], st["ring"], st["requests"], st["up_count"], st["down_count"]) == \
            (W, ref.budget, len(ref.ring), len(ref.queue), ref.up_count, ref.down_count), step
    assert steps > 10
