"""GPU parity of the KDA chunked prefill against the fp64 oracle, through the C ABI.

Tolerance: tests/_compare.py (KDA section).  Snapshot slots that the wave does not write must be
bit-identical afterwards (NaN-poisoned unread slots included).
"""
import numpy as np
import pytest
import torch

import paper_2609_35263_amd as wp
import workloads.kda as wk
from tests import _compare, _harness

pytestmark = pytest.mark.gpu


def _written(spec):
    return sorted({int(s) for s, c in zip(spec.state_out, spec.chunk_lens) if c > 0})


def check_wave(spec, seed, heads=None):
    print(f"[kda] {spec.name} seed={seed} heads={heads}", flush=True)
    t = wk.make_tensors(spec, seed)
    g = _harness.gpu_kda(spec, t)
    o_ref, pool_ref = _harness.oracle_kda(spec, t, heads=heads)
    hs = np.arange(spec.num_heads) if heads is None else np.asarray(heads)
    out = g["out"].float().cpu().numpy()[:, hs]
    reps = {"out": _compare.assert_kda_parity(out, o_ref, f"{spec.name} out")}
    pool = g["state_pool"].cpu().numpy()
    for s in _written(spec):
        reps[f"slot{s}"] = _compare.assert_kda_parity(pool[s][hs], pool_ref[s][hs], f"{spec.name} slot {s}")
    before = t["state_pool"].numpy()
    for s in range(spec.num_slots):
        if s not in _written(spec):
            assert np.array_equal(pool[s].view(np.uint32), before[s].view(np.uint32)), f"slot {s} changed"
    print(f"[kda] {spec.name}: {reps}", flush=True)
    return g, reps


def test_kda_small():
    check_wave(wk.small(), seed=101)


def test_kda_small_extreme_gates():
    """Decays with exact zeros and per-token rates up to 16: the exact pairwise path for slow channels."""
    check_wave(wk.small(extreme=True), seed=102)


def test_kda_ragged_blocks_and_single_tokens():
    spec = wk.custom(3, 128, 128, [1, 63, 65, 127, 128, 129, 2], [-1, 0, -1, 1, 2, -1, 3],
                     [4, 5, 6, 7, 8, 9, 10], 11)
    check_wave(spec, seed=103)


def test_kda_chunk_by_chunk_resume():
    """A request run as three waves, each resuming from the snapshot the previous wave wrote on the GPU,
    equals the oracle's single run."""
    H, lens = 2, [100, 37, 64]
    full = wk.custom(H, 128, 128, [sum(lens)], [0], [1], 2)
    t = wk.make_tensors(full, 104)
    o_ref, pool_ref = _harness.oracle_kda(full, t)
    pool = t["state_pool"].cuda().clone()
    outs, cu = [], 0
    for i, c in enumerate(lens):
        spec = wk.custom(H, 128, 128, [c], [0 if i == 0 else 1], [1], 2)
        part = {n: t[n][cu:cu + c] for n in ("q", "k", "v", "alpha", "beta")}
        part["state_pool"] = t["state_pool"]
        g = _harness.gpu_kda(spec, part, pool=pool)
        outs.append(g["out"].float().cpu().numpy())
        cu += c
    _compare.assert_kda_parity(np.concatenate(outs), o_ref, "chunk by chunk")
    _compare.assert_kda_parity(pool[1].cpu().numpy(), pool_ref[1], "final snapshot")


def test_kda_deterministic_and_stale_workspace():
    spec = wk.small()
    t = wk.make_tensors(spec, 105)
    g1 = _harness.gpu_kda(spec, t)
    g2 = _harness.gpu_kda(spec, t)
    assert torch.equal(g1["out"].view(torch.int16), g2["out"].view(torch.int16))
    assert torch.equal(g1["state_pool"].view(torch.int32), g2["state_pool"].view(torch.int32))
    # a workspace holding another plan's metadata: the host refuses the call, nothing is enqueued
    other = wp.kda_plan_for(wk.custom(4, 128, 128, [5], [-1], [0], 10))
    ws = wp.new_workspace(g1["plan"])
    wp.kda_upload(other, ws)
    out = torch.zeros_like(g1["out"])
    pool = t["state_pool"].cuda().clone()
    d = g1["dev"]
    with pytest.raises(wp.WaveppError) as e:
        wp.kda_chunked_prefill(g1["plan"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], pool, out, ws)
    assert e.value.status == -1 and "wavepp_kda_upload" in str(e.value)
    torch.cuda.synchronize()
    assert not out.view(torch.int16).any()
    assert torch.equal(pool.view(torch.int32), t["state_pool"].cuda().view(torch.int32))
    # the kernel's own guard: the host map names this plan, but the caller overwrote the workspace
    # header since (with the other plan's metadata): the kernel writes nothing
    wp.kda_upload(g1["plan"], ws)
    ws2 = wp.new_workspace(other)
    wp.kda_upload(other, ws2)
    n = min(ws.numel(), ws2.numel())
    ws[:n].copy_(ws2[:n])
    wp.kda_chunked_prefill(g1["plan"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], pool, out, ws)
    torch.cuda.synchronize()
    assert not out.view(torch.int16).any()
    assert torch.equal(pool.view(torch.int32), t["state_pool"].cuda().view(torch.int32))


def test_kda_idle_wave_is_a_no_op():
    spec = wk.custom(4, 128, 128, [0, 0], [0, 1], [1, 0], 2)
    t = wk.make_tensors(spec, 106)
    g = _harness.gpu_kda(spec, t)
    assert g["plan"].info()["num_items"] == 0
    assert g["out"].shape[0] == 0
    assert torch.equal(g["state_pool"].view(torch.int32).cpu(), t["state_pool"].view(torch.int32))


def test_kda_wave_full_size_sampled_heads():
    """The 16,384-token wave of four 4,096-token chunks, 64 heads; the oracle runs four heads."""
    check_wave(wk.wave(), seed=107, heads=[0, 21, 42, 63])


def test_kda_short_chunks_sampled_heads():
    check_wave(wk.short(), seed=108, heads=[5, 60])


def test_kda_long_chunk_sampled_head():
    check_wave(wk.long(), seed=109, heads=[7])


def _check_custom(spec, t, what):
    g = _harness.gpu_kda(spec, t)
    o_ref, pool_ref = _harness.oracle_kda(spec, t)
    _compare.assert_kda_parity(g["out"].float().cpu().numpy(), o_ref, f"{what} out")
    pool = g["state_pool"].cpu().numpy()
    for s in _written(spec):
        _compare.assert_kda_parity(pool[s], pool_ref[s], f"{what} slot {s}")


@pytest.mark.parametrize("case", ["no_decay", "reset_every_token", "no_write", "unit_write"])
def test_kda_degenerate_gates(case):
    """alpha = 1 (no forgetting), alpha = 0 (every channel resets every token: the exact path for all
    channels), beta = 0 (no writes: the output is the decayed snapshot read out), beta = 1."""
    spec = wk.custom(2, 128, 128, [150, 64], [0, -1], [2, 1], 3)
    t = wk.make_tensors(spec, seed=110)
    if case == "no_decay":
        t["alpha"].fill_(1.0)
    elif case == "reset_every_token":
        t["alpha"].fill_(0.0)
    elif case == "no_write":
        t["beta"].fill_(0.0)
    else:
        t["beta"].fill_(1.0)
    _check_custom(spec, t, case)


def test_kda_many_single_token_requests():
    R = 64
    spec = wk.custom(4, 128, 128, [1] * R, [i if i % 2 else -1 for i in range(R)], [R + i for i in range(R)], 2 * R)
    _check_custom(spec, wk.make_tensors(spec, seed=111), "single tokens")


def test_kda_many_heads():
    spec = wk.custom(96, 128, 128, [70, 5], [-1, 1], [0, 2], 3)
    _check_custom(spec, wk.make_tensors(spec, seed=112), "96 heads")
