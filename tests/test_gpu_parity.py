"""GPU parity of the HIP path against the fp64 oracle, through the C ABI (needs an MI355X).

Bars: append bit-exact on the whole pool; attention max-abs <= 2e-2, mean-abs <= 2e-3 on bf16 out
and LSE max-abs <= 1e-3; page permutation and repeated runs bit-identical.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from tests import _compare
from tests._harness import gpu_wave, oracle_wave, out_f64

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check_wave(spec, seed, max_splits=0, poison=True):
    torch = _torch()
    say(f"[wave] {spec.name} seed={seed} splits={max_splits} R={spec.num_requests} T={spec.total_tokens}")
    t = wl.make_tensors(spec, seed=seed, poison=poison)
    ref = oracle_wave(spec, t)
    g = gpu_wave(spec, t, max_splits=max_splits)
    assert np.array_equal(wl.to_bits(g["k_pool"]), ref["k_pool"]), "K pool after append differs"
    if not spec.kv_shared:
        assert np.array_equal(wl.to_bits(g["v_pool"]), ref["v_pool"]), "V pool after append differs"
    rep = _compare.assert_parity(out_f64(g["out"]), ref["o"], g["lse"].cpu().numpy(), ref["lse"], spec.name)
    say(f"  parity {rep}")
    return g, ref, t


def test_cfg1_full():
    check_wave(wl.cfg1(), seed=1000)


def test_cfg2_full():
    check_wave(wl.cfg2(), seed=2000)


def test_cfg2_full_four_wave_form(monkeypatch):
    """The 4-wave kernel form (128-row items, 64-key tiles, two workgroups per CU) on the whole cfg2 wave."""
    monkeypatch.setenv("WAVEPP_GQA_WAVES", "4")
    check_wave(wl.cfg2(), seed=2001)


@pytest.mark.parametrize("case", [
    # Hq, Hkv, d, B, prefix, chunk
    (8, 2, 128, 16, [48, 0, 130], [32, 7, 61]),       # d=128 on 16-token pages, p = 0, mid-page start
    (8, 2, 64, 64, [64, 5, 0], [200, 1, 129]),        # d=64 on 64-token pages, c = 1, ragged tails
    (16, 16, 128, 64, [100, 0], [33, 70]),            # MHA (G = 1)
    (16, 1, 64, 16, [37, 250], [45, 3]),              # MQA (G = 16)
    (32, 8, 128, 64, [4096, 0, 64, 700], [0, 300, 64, 129]),   # idle lane
    (24, 4, 128, 64, [200, 31], [45, 70]),            # G = 6: 32-row blocks straddle tokens at uneven rows
    (16, 4, 128, 64, [0, 40, 100, 140, 200], [20, 30, 28, 25, 30]),   # 4-wave form: 1, 2, 2, 3, 4 key tiles
    (8, 2, 64, 64, [300, 17], [25, 32]),              # 4-wave form, d = 64 on 64-token pages
    (8, 2, 128, 16, [90, 250, 0], [30, 5, 20]),       # 4-wave form, d = 128 on 16-token pages
])
def test_custom_shapes(case):
    Hq, Hkv, d, B, prefix, chunk = case
    spec = wl.custom_wave(Hq, Hkv, d, d, B, prefix, chunk, seed=sum(prefix) + d, name=f"custom{case}")
    check_wave(spec, seed=len(prefix) * 13 + B)


@pytest.mark.parametrize("splits", [1, 2, 7, 24])
def test_split_invariance_and_determinism(splits):
    """24 splits gives the longest items one split per 128-key tile (24 of them), past the merge
    kernel's single-round-trip limit of 16, and the shorter ones 16 or fewer."""
    torch = _torch()
    spec = wl.custom_wave(32, 8, 128, 128, 64, [1000, 64, 3000], [300, 129, 64], seed=9, name="split")
    g, ref, t = check_wave(spec, seed=99, max_splits=splits)
    again = gpu_wave(spec, t, max_splits=splits)
    assert torch.equal(again["out"], g["out"]) and torch.equal(again["lse"], g["lse"])


def test_page_permutation_is_bit_identical():
    torch = _torch()
    spec = wl.cfg2()
    t = wl.make_tensors(spec, seed=2001)
    g1 = gpu_wave(spec, t)
    perm = torch.as_tensor(np.random.default_rng(4).permutation(spec.num_pages))
    t2 = dict(t)
    for k in ("k_pool", "v_pool"):
        x = torch.empty_like(t[k])
        x[perm] = t[k]
        t2[k] = x
    spec2 = wl.custom_wave(32, 8, 128, 128, 64, spec.prefix_lens, spec.chunk_lens, num_pages=512)
    spec2.block_table = perm.numpy().astype(np.int32)[np.maximum(spec.block_table, 0)]
    g2 = gpu_wave(spec2, t2)
    assert torch.equal(g1["out"], g2["out"]) and torch.equal(g1["lse"], g2["lse"])


def test_chunk_by_chunk_equals_single_chunk():
    torch = _torch()
    import paper_2609_35263_amd as wp
    Hq, Hkv, d, B = 16, 4, 128, 16
    p0, chunks = 70, [33, 1, 90]
    total = sum(chunks)
    whole = wl.custom_wave(Hq, Hkv, d, d, B, [p0], [total], seed=3, bt_extra=1)
    t = wl.make_tensors(whole, seed=5)
    ref = oracle_wave(whole, t)
    dev = {k: v.cuda() for k, v in t.items()}
    outs, lses = [], []
    start, off = p0, 0
    for c in chunks:
        p = wp.plan(num_q_heads=Hq, num_kv_heads=Hkv, head_dim_qk=d, head_dim_v=d, page_size=B,
                    num_pages=whole.num_pages, softmax_scale=whole.softmax_scale, prefix_lens=[start],
                    chunk_lens=[c], block_table=whole.block_table)
        ws = wp.new_workspace(p)
        out = torch.empty((c, Hq, d), dtype=torch.bfloat16, device="cuda")
        lse = torch.empty((c, Hq), dtype=torch.float32, device="cuda")
        wp.plan_upload(p, ws)
        wp.append_kv(p, dev["k_new"][off:off + c].contiguous(), dev["v_new"][off:off + c].contiguous(),
                     dev["k_pool"], dev["v_pool"], ws)
        wp.chunked_prefill(p, dev["q"][off:off + c].contiguous(), dev["k_pool"], dev["v_pool"], out, lse, ws)
        outs.append(out)
        lses.append(lse)
        start += c
        off += c
    torch.cuda.synchronize()
    assert np.array_equal(wl.to_bits(dev["k_pool"]), ref["k_pool"])
    _compare.assert_parity(out_f64(torch.cat(outs)), ref["o"], torch.cat(lses).cpu().numpy(), ref["lse"])


def test_needles_through_permuted_pages():
    torch = _torch()
    spec = wl.custom_wave(8, 2, 128, 128, 16, [96, 40], [50, 30], seed=12)
    t = wl.make_tensors(spec, seed=12)
    rng = np.random.default_rng(2)
    u = rng.standard_normal(128)
    u /= np.linalg.norm(u)
    t["q"][:] = torch.as_tensor(u * 3.0, dtype=torch.float32).to(torch.bfloat16)
    kn = t["k_new"].float()
    kp = t["k_pool"].float()
    for r in range(2):
        p, c = int(spec.prefix_lens[r]), int(spec.chunk_lens[r])
        cu = int(spec.cu_tokens[r])
        pos = sorted({j for b in range((p + c + 15) // 16) for j in (16 * b, 16 * b + 15) if j < p + c}
                     | {p - 1, p, p + c - 1})
        for rank, j in enumerate(pos):
            vec = torch.as_tensor(u * (5.0 * (rank + 1) / 3.0 / spec.softmax_scale), dtype=torch.float32)
            if j >= p:
                kn[cu + j - p, :] = vec
            else:
                kp[int(spec.block_table[r, j // 16]), :, j % 16] = vec
    t["k_new"] = kn.to(torch.bfloat16)
    kp = kp.to(torch.bfloat16)
    t["k_pool"] = kp
    ref = oracle_wave(spec, t)
    g = gpu_wave(spec, t)
    _compare.assert_parity(out_f64(g["out"]), ref["o"], g["lse"].cpu().numpy(), ref["lse"], "needles")


def test_idle_wave_is_a_no_op():
    """A wave whose requests all have empty chunks (c_r = 0): every entry point returns OK and the
    pools are left as they were."""
    spec = wl.custom_wave(8, 2, 64, 64, 16, [48, 0, 130], [0, 0, 0], seed=3)
    t = wl.make_tensors(spec, seed=3, poison=True)
    before = {k: wl.to_bits(t[k]) for k in ("k_pool", "v_pool")}
    g = gpu_wave(spec, t)
    assert g["plan"].info()["num_items"] == 0 and g["out"].shape[0] == 0
    for k in ("k_pool", "v_pool"):
        assert np.array_equal(wl.to_bits(g[k]), before[k]), k


def test_single_visible_key_is_bit_exact():
    torch = _torch()
    spec = wl.custom_wave(8, 2, 64, 64, 16, [0, 0], [1, 1], seed=1)
    t = wl.make_tensors(spec, seed=1)
    g = gpu_wave(spec, t)
    for tok in range(2):
        for h in range(8):
            assert torch.equal(g["out"][tok, h].cpu(), t["v_new"][tok, h // 4])


def test_wrong_workspace_or_small_workspace():
    torch = _torch()
    import paper_2609_35263_amd as wp
    spec = wl.custom_wave(8, 2, 64, 64, 16, [500], [32], seed=3)
    t = wl.make_tensors(spec, seed=1000)
    p = wp.plan_for(spec, max_splits=2)
    assert p.workspace_bytes > 256                  # split partials need workspace beyond the metadata
    small = torch.empty(p.workspace_bytes - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(wp.WaveppError) as e:
        wp.plan_upload(p, small)
    assert e.value.status == -6
    # a workspace holding another plan's metadata: the host refuses the calls, nothing is enqueued
    other = wp.plan_for(spec, max_splits=2)
    ws = wp.new_workspace(p)
    wp.plan_upload(other, ws)
    out = torch.full((spec.total_tokens, 8, 64), 7.0, dtype=torch.bfloat16, device="cuda")
    d = {k: v.cuda() for k, v in t.items()}
    with pytest.raises(wp.WaveppError) as e:
        wp.chunked_prefill(p, d["q"], d["k_pool"], d["v_pool"], out, None, ws)
    assert e.value.status == -1 and "wavepp_attn_plan_upload" in str(e.value)
    with pytest.raises(wp.WaveppError) as e:
        wp.append_kv(p, d["k_new"], d["v_new"], d["k_pool"], d["v_pool"], ws)
    assert e.value.status == -1
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    # the kernels' own guard: the host map says this plan, but the workspace header was overwritten
    # since (here by the other plan's metadata, copied in by the caller): the kernels write nothing
    wp.plan_upload(p, ws)
    ws2 = wp.new_workspace(other)
    wp.plan_upload(other, ws2)
    n = min(ws.numel(), ws2.numel())
    ws[:n].copy_(ws2[:n])
    wp.chunked_prefill(p, d["q"], d["k_pool"], d["v_pool"], out, None, ws)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    # and after a proper upload the same call runs
    wp.plan_upload(p, ws)
    wp.append_kv(p, d["k_new"], d["v_new"], d["k_pool"], d["v_pool"], ws)
    wp.chunked_prefill(p, d["q"], d["k_pool"], d["v_pool"], out, None, ws)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out.float()).all())


def test_sampled_rows_cfg3():
    sampled_config_check(wl.cfg3(), seed=3000)


def test_sampled_rows_cfg4_all_four_layers():
    """The concurrency-128 wave as the bench runs it: one plan and one upload, then append and
    attention for four layers with distinct pools, queries and outputs; sampled rows of every layer
    against the oracle, and every layer's pools bit-exact."""
    torch = _torch()
    import paper_2609_35263_amd as wp
    spec = wl.cfg4()
    assert spec.layers == 4
    say(f"[layers] {spec.name} R={spec.num_requests} T={spec.total_tokens} layers={spec.layers}")
    samples = sample_rows(spec, seed=4000)
    p = wp.plan_for(spec)
    ws = wp.new_workspace(p)
    wp.plan_upload(p, ws)
    layers, refs = [], []
    for l in range(spec.layers):
        t = wl.make_tensors(spec, seed=4000, device="cuda", poison=True, layer=l)
        refs.append(oracle_rows(spec, t, samples))
        out = torch.full((spec.total_tokens, spec.num_q_heads, spec.head_dim_v), float("nan"), dtype=torch.bfloat16,
                         device="cuda")
        lse = torch.full((spec.total_tokens, spec.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
        layers.append((t, out, lse))
    for t, out, lse in layers:
        wp.append_kv(p, t["k_new"], t["v_new"], t["k_pool"], t["v_pool"], ws)
        wp.chunked_prefill(p, t["q"], t["k_pool"], t["v_pool"], out, lse, ws)
    torch.cuda.synchronize()
    for l, ((t, out, lse), ref) in enumerate(zip(layers, refs)):
        o = out_f64(out[samples[:, 0], samples[:, 1]])
        ls = lse[samples[:, 0], samples[:, 1]].cpu().numpy()
        rep = _compare.assert_parity(o, ref["o"], ls, ref["lse"], f"{spec.name} layer {l}")
        assert bool(torch.isfinite(out.float()).all()), f"non-finite output in layer {l}"
        assert np.array_equal(wl.to_bits(t["k_pool"]), ref["k_pool"]), f"K pool of layer {l}"
        assert np.array_equal(wl.to_bits(t["v_pool"]), ref["v_pool"]), f"V pool of layer {l}"
        say(f"  layer {l} parity {rep} over {len(samples)} rows")
    # the layers differ: a kernel that read layer 0's pools for every layer would be caught here
    assert not np.array_equal(refs[0]["o"], refs[1]["o"])


def test_sampled_rows_cfg6p():
    """The paper's 4K-suffix-behind-125K-prefix wave."""
    sampled_config_check(wl.cfg6p(), seed=6000, rows_per_req=12)


@pytest.mark.parametrize("chunk", [16, 32, 64, 128])
def test_sampled_rows_small_chunk_wave(chunk):
    """Short chunks over 16K-32K cached tokens (the gather-bound sweep): 128-row items with 64-key
    tiles at c = 16, 256-row items beyond; automatic key-range splits and the merge."""
    sampled_config_check(wl.small_chunk(chunk), seed=7000 + chunk)


def sample_rows(spec, seed, rows_per_req=16, heads_per_row=4):
    """(packed token, query head) rows of every request with a chunk: the first and last chunk token,
    the tokens on either side of every page boundary the chunk crosses (at most 8 of them), and seeded
    random tokens, each with `heads_per_row` random heads; plus one random token with every head."""
    rng = np.random.default_rng(seed)
    cu = spec.cu_tokens
    B = spec.page_size
    samples = set()
    for r in range(spec.num_requests):
        p, c = int(spec.prefix_lens[r]), int(spec.chunk_lens[r])
        if c == 0:
            continue
        toks = {0, c - 1}
        bounds = [i for i in range(c) if (p + i) % B == 0][:4]
        for i in bounds:
            toks |= {max(0, i - 1), i}
        toks |= set(rng.integers(0, c, rows_per_req).tolist())
        for i in toks:
            for h in rng.choice(spec.num_q_heads, min(heads_per_row, spec.num_q_heads), replace=False):
                samples.add((int(cu[r]) + int(i), int(h)))
        full = int(rng.integers(0, c))
        for h in range(spec.num_q_heads):
            samples.add((int(cu[r]) + full, h))
    return np.array(sorted(samples))


def oracle_rows(spec, t, samples):
    """Oracle append (whole pools, bit patterns) and attention of the sampled rows, from copies of the
    inputs taken before the HIP path runs."""
    q_rows = {int(tok): wl.to_bits(t["q"][int(tok)]) for tok in set(samples[:, 0].tolist())}
    pools_before = {k: wl.to_bits(t[k]) for k in ("k_pool", "v_pool") if t[k] is not None}
    new = {k: wl.to_bits(t[k]) for k in ("k_new", "v_new") if t[k] is not None}
    k1, v1 = oracle.append_kv(pools_before["k_pool"], pools_before.get("v_pool"), new["k_new"], new.get("v_new"),
                              spec.prefix_lens, spec.chunk_lens, spec.block_table, spec.page_size)
    o_ref, l_ref = oracle.chunked_prefill_rows(q_rows, k1, v1, spec.prefix_lens, spec.chunk_lens, spec.block_table,
                                               samples, page_size=spec.page_size, num_kv_heads=spec.num_kv_heads,
                                               softmax_scale=spec.softmax_scale, kv_shared=spec.kv_shared,
                                               head_dim_v=spec.head_dim_v)
    return {"o": o_ref, "lse": l_ref, "k_pool": k1, "v_pool": v1}


def sampled_config_check(spec, seed, rows_per_req=16, heads_per_row=4):
    """Large configs: the full HIP path runs; the oracle recomputes sampled rows of every request."""
    torch = _torch()
    say(f"[sampled] {spec.name} R={spec.num_requests} T={spec.total_tokens}")
    t = wl.make_tensors(spec, seed=seed, device="cuda", poison=True)
    samples = sample_rows(spec, seed, rows_per_req, heads_per_row)
    ref = oracle_rows(spec, t, samples)
    g = gpu_wave(spec, t)
    o = out_f64(g["out"][samples[:, 0], samples[:, 1]])
    lse = g["lse"][samples[:, 0], samples[:, 1]].cpu().numpy()
    rep = _compare.assert_parity(o, ref["o"], lse, ref["lse"], spec.name)
    assert bool(torch.isfinite(g["out"].float()).all()), "non-finite output"
    assert np.array_equal(wl.to_bits(g["k_pool"]), ref["k_pool"])
    if ref["v_pool"] is not None:
        assert np.array_equal(wl.to_bits(g["v_pool"]), ref["v_pool"])
    reqs = set(np.searchsorted(spec.cu_tokens, samples[:, 0], side="right") - 1)
    say(f"  parity {rep} over {len(samples)} rows of {len(reqs)} requests")
    return len(reqs)


# ------------------------------------------------------------------------------------------
# Latent (MLA, absorbed) attention: one shared 576-wide latent, values = its first 512 lanes
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("case", [
    # Hq, B, prefix, chunk
    (16, 64, [130, 0], [70, 33]),
    (128, 64, [64], [3]),
    (8, 16, [37, 200, 5], [20, 1, 90]),
    (40, 64, [100, 3], [17, 50]),      # G = 40: rows of one 32-row block belong to two tokens
    (96, 64, [64, 129], [5, 2]),       # G = 96: a 128-row item spans two tokens
])
def test_latent_small(case):
    Hq, B, prefix, chunk = case
    spec = wl.custom_wave(Hq, 1, 576, 512, B, prefix, chunk, kv_shared=True, seed=sum(prefix) + Hq,
                          name=f"latent{case}")
    check_wave(spec, seed=len(prefix) + B)


@pytest.mark.parametrize("splits", [2, 3])
def test_latent_splits(splits):
    spec = wl.custom_wave(16, 1, 576, 512, 64, [700, 64], [40, 129], kv_shared=True, seed=77, name="latent_split")
    check_wave(spec, seed=78, max_splits=splits)


@pytest.mark.parametrize("chunk", [10, 40])   # 40 rows: the 4-wave form; 160 rows: the 8-wave form
def test_grouped_reference_overflow_takes_exact_second_pass(chunk):
    # a key in a later tile has a logit ~159 (log2 units) above everything in the first tile, so the
    # first pass's fixed per-row reference overflows and the workgroup redoes the item exactly
    torch = _torch()
    spec = wl.custom_wave(8, 2, 128, 128, 64, [300], [chunk], seed=15, name=f"grouped_ovf{chunk}")
    t = wl.make_tensors(spec, seed=16)
    rng = np.random.default_rng(4)
    u = rng.standard_normal(128)
    u /= np.linalg.norm(u)
    t["q"][:] = torch.as_tensor(u * 2.0, dtype=torch.float32).to(torch.bfloat16)
    kp = t["k_pool"].float()
    j = 250
    for g in range(2):
        kp[int(spec.block_table[0, j // 64]), g, j % 64] = torch.as_tensor(u * (110.0 / 2.0 / spec.softmax_scale),
                                                                             dtype=torch.float32)
    t["k_pool"] = kp.to(torch.bfloat16)
    ref = oracle_wave(spec, t)
    g = gpu_wave(spec, t)
    _compare.assert_parity(out_f64(g["out"]), ref["o"], g["lse"].cpu().numpy(), ref["lse"], f"grouped overflow {chunk}")


def test_latent_reference_overflow_takes_exact_second_pass():
    # a key far later in the sequence has a logit ~150 (log2 units) above everything in the first
    # tile, so the fixed per-row reference is exceeded and the workgroup redoes its key range
    torch = _torch()
    spec = wl.custom_wave(16, 1, 576, 512, 64, [300], [10], kv_shared=True, seed=5, name="latent_ovf")
    t = wl.make_tensors(spec, seed=6)
    rng = np.random.default_rng(3)
    u = rng.standard_normal(576)
    u /= np.linalg.norm(u)
    t["q"][:] = torch.as_tensor(u * 2.0, dtype=torch.float32).to(torch.bfloat16)
    kp = t["k_pool"].float()
    j = 250
    kp[int(spec.block_table[0, j // 64]), 0, j % 64] = torch.as_tensor(u * (110.0 / 2.0 / spec.softmax_scale),
                                                                         dtype=torch.float32)
    t["k_pool"] = kp.to(torch.bfloat16)
    ref = oracle_wave(spec, t)
    g = gpu_wave(spec, t)
    _compare.assert_parity(out_f64(g["out"]), ref["o"], g["lse"].cpu().numpy(), ref["lse"], "latent overflow")


def test_sampled_rows_cfg5():
    """The latent wave: sampled rows of all 8 requests (each over 139K visible keys)."""
    n = sampled_config_check(wl.cfg5(), seed=5000, rows_per_req=8, heads_per_row=3)
    assert n == 8
