"""The allocation-free entry point (wavepp_attn_chunked_prefill_noalloc) against the workspace entry
points, through the C ABI, on consecutive calls that share the static scratch: each call's pools,
output and LSE must be bit-identical to wavepp_attn_append_kv + wavepp_attn_chunked_prefill on the
same plan and inputs, and within the oracle's tolerance.  The calls shrink (a split GQA wave, then a
smaller split latent wave, then the smallest wave), so a result that depended on scratch left over
from an earlier call would show up.
"""
import numpy as np
import pytest

import workloads as wl
from tests import _compare
from tests._harness import gpu_wave, oracle_wave, out_f64

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _noalloc_wave(spec, t, max_splits):
    torch = _torch()
    import paper_2609_35263_amd as wp
    d = {k: (None if v is None else v.to("cuda").contiguous()) for k, v in t.items()}
    p = wp.plan_for(spec, max_splits=max_splits)
    T = spec.total_tokens
    out = torch.full((T, spec.num_q_heads, spec.head_dim_v), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((T, spec.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
    wp.chunked_prefill_noalloc(p, d["q"], d["k_pool"], d["v_pool"], out, lse, k_new=d["k_new"], v_new=d["v_new"])
    torch.cuda.synchronize()
    return {"k_pool": d["k_pool"], "v_pool": d["v_pool"], "out": out, "lse": lse, "plan": p}


@pytest.mark.parametrize("case", ["gqa_split", "latent_split", "cfg1"])
def test_noalloc_matches_workspace_entry_points(case):
    torch = _torch()
    if case == "gqa_split":
        spec = wl.custom_wave(32, 8, 128, 128, 64, [1000, 64, 3000], [300, 129, 64], seed=9, name="noalloc_gqa")
        splits, seed = 3, 91
    elif case == "latent_split":
        spec = wl.custom_wave(16, 1, 576, 512, 64, [700, 64], [40, 129], kv_shared=True, seed=77, name="noalloc_mla")
        splits, seed = 2, 92
    else:
        spec, splits, seed = wl.cfg1(), 0, 93
    print(f"[noalloc] {case} R={spec.num_requests} T={spec.total_tokens} splits={splits}", flush=True)
    t = wl.make_tensors(spec, seed=seed, poison=True)
    ref = oracle_wave(spec, t)
    a = gpu_wave(spec, t, max_splits=splits)
    b = _noalloc_wave(spec, t, splits)
    if splits:
        assert b["plan"].info()["num_merge_items"] > 0, "the case must exercise split partials in the scratch"
    for k in ("k_pool", "v_pool"):
        if a[k] is not None:
            # bit patterns: the unused pool slots hold NaN
            assert torch.equal(a[k].view(torch.int16), b[k].view(torch.int16)), f"{k} after the append differs"
            assert np.array_equal(wl.to_bits(b[k]), ref[k]), f"{k} after the append is not the oracle's"
    assert torch.equal(a["out"].view(torch.int16), b["out"].view(torch.int16)), "output differs"
    assert torch.equal(a["lse"].view(torch.int32), b["lse"].view(torch.int32)), "LSE differs"
    rep = _compare.assert_parity(out_f64(b["out"]), ref["o"], b["lse"].cpu().numpy(), ref["lse"], case)
    print(f"  noalloc {case}: bit-identical to the workspace path; parity {rep}", flush=True)


@pytest.mark.parametrize("case", ["gqa_split", "latent_split"])
def test_noalloc_graph_replays_match_eager(case):
    """The allocation-free entry point under HIP stream capture: the wave's append and attention are
    captured once and replayed three times, with eager work on the same tensors and a synchronization
    between replays; every replay must leave the pools, output and LSE bit-identical to an eager call
    of the same entry point on the same plan."""
    torch = _torch()
    import paper_2609_35263_amd as wp
    if case == "gqa_split":
        spec = wl.custom_wave(32, 8, 128, 128, 64, [1000, 64, 3000], [300, 129, 64], seed=9, name="graph_gqa")
        splits, seed = 3, 94
    else:
        spec = wl.custom_wave(16, 1, 576, 512, 64, [700, 64], [40, 129], kv_shared=True, seed=77, name="graph_mla")
        splits, seed = 2, 95
    print(f"[graph noalloc] {case} R={spec.num_requests} T={spec.total_tokens} splits={splits}", flush=True)
    t = wl.make_tensors(spec, seed=seed, poison=True)
    d = {k: (None if v is None else v.to("cuda").contiguous()) for k, v in t.items()}
    p = wp.plan_for(spec, max_splits=splits)
    assert p.info()["num_merge_items"] > 0
    T = spec.total_tokens
    # eager reference on copies of the pools
    kp_e = d["k_pool"].clone()
    vp_e = None if d["v_pool"] is None else d["v_pool"].clone()
    out_e = torch.empty((T, spec.num_q_heads, spec.head_dim_v), dtype=torch.bfloat16, device="cuda")
    lse_e = torch.empty((T, spec.num_q_heads), dtype=torch.float32, device="cuda")
    wp.chunked_prefill_noalloc(p, d["q"], kp_e, vp_e, out_e, lse_e, k_new=d["k_new"], v_new=d["v_new"])
    torch.cuda.synchronize()
    # captured call on the original pools
    out = torch.empty_like(out_e)
    lse = torch.empty_like(lse_e)
    kp, vp = d["k_pool"], d["v_pool"]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        wp.chunked_prefill_noalloc(p, d["q"], kp, vp, out, lse, k_new=d["k_new"], v_new=d["v_new"])
    torch.cuda.synchronize()
    for rep in range(3):
        # eager work between replays: clear the outputs (a fill kernel, not a memset node in the graph)
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(kp.view(torch.int16), kp_e.view(torch.int16)), f"replay {rep}: k_pool differs"
        if vp is not None:
            assert torch.equal(vp.view(torch.int16), vp_e.view(torch.int16)), f"replay {rep}: v_pool differs"
        assert torch.equal(out.view(torch.int16), out_e.view(torch.int16)), f"replay {rep}: output differs"
        assert torch.equal(lse.view(torch.int32), lse_e.view(torch.int32)), f"replay {rep}: LSE differs"
        print(f"  replay {rep}: bit-identical to the eager call", flush=True)
    del g
