"""Host-side checks of the KDA entry points that need no GPU: validation, work list, tolerance teeth."""
import numpy as np
import pytest
import torch

import paper_2609_35263_amd as wp
import workloads as wl
import workloads.kda as wk
from oracle import kda as ok
from tests import _compare


def kw(**over):
    base = dict(num_heads=4, head_dim_k=128, head_dim_v=128, num_state_slots=6, chunk_lens=[40, 0, 130],
                state_in=[-1, 5, 0], state_out=[1, 2, 0])
    base.update(over)
    return base


def status_of(**over):
    try:
        wp.kda_plan(**kw(**over))
        return 0
    except wp.WaveppError as e:
        return e.status


def test_valid_plan_orders_longest_first():
    p = wp.kda_plan(**kw())
    info = p.info()
    assert info["total_tokens"] == 170
    assert info["num_items"] == 2            # the idle lane is dropped
    assert info["block_tokens"] == 64
    assert info["workspace_bytes"] % 256 == 0 and info["workspace_bytes"] >= info["metadata_bytes"]


@pytest.mark.parametrize("over,status", [
    (dict(head_dim_k=64, head_dim_v=64), -2),
    (dict(head_dim_v=64), -2),
    (dict(num_heads=0), -1),
    (dict(chunk_lens=[40, -1, 130]), -1),
    (dict(state_in=[6, 5, 0]), -3),            # outside the pool
    (dict(state_in=[-2, 5, 0]), -3),
    (dict(state_out=[-1, 2, 0]), -3),          # an active request must write a slot
    (dict(state_out=[0, 2, 0]), -4),           # two requests write slot 0
    (dict(state_in=[0, 5, 3], state_out=[1, 2, 0]), -4),   # request 0 resumes from what request 2 writes
    (dict(chunk_lens=[40], state_in=[-1], state_out=[1, 2]), "value"),
])
def test_invalid_waves_are_rejected(over, status):
    if status == "value":
        with pytest.raises(ValueError):
            wp.kda_plan(**kw(**over))
    else:
        assert status_of(**over) == status


def test_accepted_edge_cases():
    assert status_of(state_in=[1, 5, 0], state_out=[1, 2, 0]) == 0          # resume in place
    assert status_of(chunk_lens=[0, 0, 0], state_in=[9, 9, 9], state_out=[-5, 9, 9]) == 0   # idle slots unchecked
    assert status_of(chunk_lens=[], state_in=[], state_out=[]) == 0
    assert status_of(chunk_lens=[1, 0, 1], state_out=[1, 1, 0]) == 0        # the idle lane's slot is not written
    p = wp.kda_plan(**kw(chunk_lens=[0, 0, 0]))
    assert p.info()["num_items"] == 0 and p.info()["total_tokens"] == 0


def test_workload_specs_are_valid():
    for name in ["kda_small", "kda_small_extreme", "kda_wave", "kda_long", "kda_short"]:
        spec = wk.config(name)
        p = wp.kda_plan_for(spec)
        assert p.info()["total_tokens"] == spec.total_tokens


# ------------------------------------------------------------------------------------------------
# Teeth of the KDA tolerance: plausible kernel mistakes, planted in the oracle on the CPU, must fail.
# ------------------------------------------------------------------------------------------------

def _small_case(seed=11, H=2, c=200):
    spec = wk.custom(H, 128, 128, [c], [0], [1], 2)
    t = wk.make_tensors(spec, seed)
    bits = {n: wl.to_bits(t[n]) for n in ("q", "k", "v")}
    return spec, t, bits


def _run(bits, t, alpha=None, beta=None, pool=None, state_in=(0,)):
    return ok.chunked_prefill(bits["q"], bits["k"], bits["v"], t["alpha"].numpy() if alpha is None else alpha,
                              t["beta"].numpy() if beta is None else beta,
                              t["state_pool"].numpy() if pool is None else pool, [bits["q"].shape[0]],
                              list(state_in), [1])


def test_tolerance_accepts_bf16_rounding_of_the_exact_result():
    spec, t, bits = _small_case()
    o, pool = _run(bits, t)
    o_bf = torch.as_tensor(o).to(torch.bfloat16).double().numpy()
    assert _compare.kda_report(o_bf, o)["ok"]


@pytest.mark.parametrize("mistake", ["drop_token", "decay_shifted", "beta_ignored", "cold_start",
                                     "block_boundary_state_lost"])
def test_tolerance_rejects_planted_mistakes(mistake):
    spec, t, bits = _small_case()
    o, pool = _run(bits, t)
    alpha, beta = t["alpha"].numpy().copy(), t["beta"].numpy().copy()
    if mistake == "drop_token":
        beta[70] = 0.0
        bits = dict(bits)
        k = bits["k"].copy()
        k[70] = 0
        bits["k"] = k
        o2, _ = _run(bits, t, beta=beta)
    elif mistake == "decay_shifted":
        alpha = np.concatenate([np.ones_like(alpha[:1]), alpha[:-1]])
        o2, _ = _run(bits, t, alpha=alpha)
    elif mistake == "beta_ignored":
        o2, _ = _run(bits, t, beta=np.ones_like(beta))
    elif mistake == "cold_start":
        o2, _ = _run(bits, t, state_in=(-1,))
    else:
        # the state is lost at the 64-token block boundary: tokens from 64 on start from zero
        o_a, _ = ok.chunked_prefill(bits["q"][:64], bits["k"][:64], bits["v"][:64], alpha[:64], beta[:64],
                                    t["state_pool"].numpy(), [64], [0], [1])
        o_b, _ = ok.chunked_prefill(bits["q"][64:], bits["k"][64:], bits["v"][64:], alpha[64:], beta[64:],
                                    t["state_pool"].numpy(), [136], [-1], [1])
        o2 = np.concatenate([o_a, o_b])
    assert not _compare.kda_report(o2, o)["ok"], mistake


# The same teeth at the size of one request of the measured KDA wave: a 4,096-token chunk resumed
# from a snapshot, with heads spread over the decay rates the wave draws.  A mistake confined to one
# 64-token block, or a decay applied one token late, must still fail the bar over the whole chunk.
_WAVE_CASE = {}


def _wave_case():
    if not _WAVE_CASE:
        spec = wk.custom(4, 128, 128, [4096], [0], [1], 2, name="kda_wave_request")
        t = wk.make_tensors(spec, seed=4040)
        bits = {n: wl.to_bits(t[n]) for n in ("q", "k", "v")}
        o, _ = _run(bits, t)
        _WAVE_CASE.update(spec=spec, t=t, bits=bits, o=o)
    return _WAVE_CASE


@pytest.mark.parametrize("mistake", ["decay_one_token_late", "block_dropped", "resume_from_zero"])
def test_tolerance_rejects_planted_mistakes_at_wave_size(mistake):
    case = _wave_case()
    t, bits, o = case["t"], case["bits"], case["o"]
    assert _compare.kda_scale(o) <= 1.5          # outputs of order one: the bar is (nearly) the unscaled one
    alpha, beta = t["alpha"].numpy().copy(), t["beta"].numpy().copy()
    if mistake == "decay_one_token_late":
        # token t's state is decayed by alpha_{t-1} (the first token by none)
        o2, _ = _run(bits, t, alpha=np.concatenate([np.ones_like(alpha[:1]), alpha[:-1]]))
    elif mistake == "block_dropped":
        # the updates of tokens 2048..2111 (one 64-token block in the middle) never reach the state
        alpha[2048:2112] = 1.0
        beta[2048:2112] = 0.0
        o2, _ = _run(bits, t, alpha=alpha, beta=beta)
    else:
        o2, _ = _run(bits, t, state_in=(-1,))
    rep = _compare.kda_report(o2, o)
    assert not rep["ok"], (mistake, rep)
