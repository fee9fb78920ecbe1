"""Run one wave through the HIP path and through the oracle on the same seeded inputs."""
import numpy as np

import oracle
import workloads as wl


def oracle_wave(spec, t):
    """Oracle append then attention on CPU copies of the inputs; returns dict of numpy arrays."""
    bits = {k: wl.to_bits(v) for k, v in t.items()}
    k1, v1 = oracle.append_kv(bits["k_pool"], bits["v_pool"], bits["k_new"], bits["v_new"], spec.prefix_lens,
                              spec.chunk_lens, spec.block_table, spec.page_size)
    o, lse = oracle.chunked_prefill(bits["q"], k1, v1, spec.prefix_lens, spec.chunk_lens, spec.block_table,
                                    page_size=spec.page_size, num_kv_heads=spec.num_kv_heads,
                                    softmax_scale=spec.softmax_scale, kv_shared=spec.kv_shared,
                                    head_dim_v=spec.head_dim_v)
    return {"k_pool": k1, "v_pool": v1, "o": o, "lse": lse}


def gpu_wave(spec, t, max_splits=0, device="cuda", with_lse=True, plan=None):
    """HIP path: plan, upload, append, attention.  Inputs are copied to the device first; the
    returned dict holds device tensors (pools after the append, out, lse)."""
    import torch
    import paper_2609_35263_amd as wp
    d = {k: (None if v is None else v.to(device).contiguous()) for k, v in t.items()}
    p = plan or wp.plan_for(spec, max_splits=max_splits)
    ws = wp.new_workspace(p, device)
    T = spec.total_tokens
    out = torch.full((T, spec.num_q_heads, spec.head_dim_v), float("nan"), dtype=torch.bfloat16, device=device)
    lse = torch.full((T, spec.num_q_heads), float("nan"), dtype=torch.float32, device=device) if with_lse else None
    wp.plan_upload(p, ws)
    wp.append_kv(p, d["k_new"], d["v_new"], d["k_pool"], d["v_pool"], ws)
    wp.chunked_prefill(p, d["q"], d["k_pool"], d["v_pool"], out, lse, ws)
    torch.cuda.synchronize()
    return {"k_pool": d["k_pool"], "v_pool": d["v_pool"], "out": out, "lse": lse, "plan": p, "ws": ws, "dev": d}


def out_f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


# ------------------------------------------------------------------------------------------------
# KDA chunked prefill
# ------------------------------------------------------------------------------------------------

def oracle_kda(spec, t, heads=None):
    """Oracle KDA wave on CPU copies of the inputs: (o [T, len(heads), d_v], pool_after [slots, H, d_k, d_v])."""
    bits = {n: wl.to_bits(t[n]) for n in ("q", "k", "v")}
    return oracle.kda.chunked_prefill(bits["q"], bits["k"], bits["v"], t["alpha"].cpu().numpy(),
                                      t["beta"].cpu().numpy(), t["state_pool"].cpu().numpy(), spec.chunk_lens,
                                      spec.state_in, spec.state_out, heads=heads)


def gpu_kda(spec, t, device="cuda", plan=None, pool=None):
    """HIP path: plan, upload, chunked prefill.  Returns device tensors (out, state_pool)."""
    import torch
    import paper_2609_35263_amd as wp
    d = {n: t[n].to(device).contiguous() for n in ("q", "k", "v", "alpha", "beta")}
    pool = t["state_pool"].to(device).contiguous().clone() if pool is None else pool
    p = plan or wp.kda_plan_for(spec)
    ws = wp.new_workspace(p, device)
    out = torch.full((spec.total_tokens, spec.num_heads, spec.head_dim_v), float("nan"), dtype=torch.bfloat16,
                     device=device)
    wp.kda_upload(p, ws)
    wp.kda_chunked_prefill(p, d["q"], d["k"], d["v"], d["alpha"], d["beta"], pool, out, ws)
    torch.cuda.synchronize()
    return {"out": out, "state_pool": pool, "plan": p, "ws": ws, "dev": d}
