"""End-to-end on the GPU: the rows working together as the paper composes them.

A first request is served cold, in chunks, leaving its K/V in pages and KDA snapshots at its chunk
boundaries.  Its block hashes and snapshot boundaries go into the hint index.  Four more requests
then find their reusable prefix (gallop/bisect over the attention blocks, then the backward scan to a
snapshot), share the cached pages and resume from the snapshot, and have their suffixes chunked into
waves by the MPU planner.  Each wave runs the append, the paged attention and the KDA chunked prefill
through the C ABI.  Every output row is compared with the oracles run over each request's whole
prompt from scratch, so a wrong reuse endpoint, page, span or snapshot shows up as a mismatch.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_35263_amd as wp
from oracle import kda as okda
from tests import _compare

pytestmark = pytest.mark.gpu

B = 16                      # page size = hashed block size
HQ, HKV, D = 4, 2, 64       # attention layer
HK, DK = 2, 128             # KDA layer
SCALE = 1.0 / 8.0


def bf16(x):
    return torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)


class Request:
    """Per-position inputs of one prompt; positions shared with another prompt copy its inputs (the
    same tokens at the same positions give the same projections)."""

    def __init__(self, rng, n, base=None, shared=0):
        self.n = n
        self.tokens = rng.integers(0, 50000, n)
        self.q = rng.standard_normal((n, HQ, D)).astype(np.float32)
        self.k = rng.standard_normal((n, HKV, D)).astype(np.float32)
        self.v = rng.standard_normal((n, HKV, D)).astype(np.float32)
        kq = rng.standard_normal((n, HK, DK)).astype(np.float32)
        self.kq = kq / np.linalg.norm(kq, axis=-1, keepdims=True)
        kk = rng.standard_normal((n, HK, DK)).astype(np.float32)
        self.kk = kk / np.linalg.norm(kk, axis=-1, keepdims=True)
        self.kv = rng.standard_normal((n, HK, DK)).astype(np.float32)
        self.alpha = np.exp(-0.05 * np.log1p(np.exp(rng.standard_normal((n, HK, DK))))).astype(np.float32)
        self.beta = (1.0 / (1.0 + np.exp(-rng.standard_normal((n, HK))))).astype(np.float32)
        if base is not None and shared:
            for name in ("tokens", "q", "k", "v", "kq", "kk", "kv", "alpha", "beta"):
                getattr(self, name)[:shared] = getattr(base, name)[:shared]
        # bf16-exact inputs for both sides
        for name in ("q", "k", "v", "kq", "kk", "kv"):
            setattr(self, name, bf16(getattr(self, name)).float().numpy())
        self.table = []             # block table (physical pages)
        self.slot = None            # KDA snapshot slot holding its current state
        self.out_attn = np.full((n, HQ, D), np.nan)
        self.out_kda = np.full((n, HK, DK), np.nan)


class Cache:
    def __init__(self, num_pages, num_slots, dev):
        self.k_pool = torch.zeros((num_pages, HKV, B, D), dtype=torch.bfloat16, device=dev)
        self.v_pool = torch.zeros_like(self.k_pool)
        self.state_pool = torch.zeros((num_slots, HK, DK, DK), dtype=torch.float32, device=dev)
        self.free_pages = list(range(num_pages))
        self.free_slots = list(range(num_slots))

    def page(self):
        return self.free_pages.pop(0)

    def slot(self):
        return self.free_slots.pop(0)


def run_wave(cache, reqs, spans, dev, snapshot_each_chunk=False):
    """One wave: append + attention and KDA for spans (request index, start, length)."""
    # pages for the new positions
    for ri, start, length in spans:
        r = reqs[ri]
        while len(r.table) * B < start + length:
            r.table.append(cache.page())
    stride = max(len(reqs[ri].table) for ri, _, _ in spans)
    bt = np.full((len(spans), stride), -1, np.int32)
    for i, (ri, _, _) in enumerate(spans):
        bt[i, :len(reqs[ri].table)] = reqs[ri].table
    prefix = np.array([s for _, s, _ in spans], np.int32)
    chunk = np.array([l for _, _, l in spans], np.int32)
    cat = lambda name: torch.cat([bf16(getattr(reqs[ri], name)[s:s + l]) for ri, s, l in spans]).to(dev).contiguous()
    p = wp.plan(num_q_heads=HQ, num_kv_heads=HKV, head_dim_qk=D, head_dim_v=D, page_size=B,
                num_pages=cache.k_pool.shape[0], softmax_scale=SCALE, prefix_lens=prefix, chunk_lens=chunk,
                block_table=bt)
    ws = wp.new_workspace(p, dev)
    T = int(chunk.sum())
    out = torch.empty((T, HQ, D), dtype=torch.bfloat16, device=dev)
    wp.plan_upload(p, ws)
    wp.append_kv(p, cat("k"), cat("v"), cache.k_pool, cache.v_pool, ws)
    wp.chunked_prefill(p, cat("q"), cache.k_pool, cache.v_pool, out, None, ws)
    # KDA: resume from each request's current slot; the first chunk writes a slot of its own
    s_in, s_out = [], []
    for ri, _, _ in spans:
        r = reqs[ri]
        s_in.append(-1 if r.slot is None else r.slot)
        if r.slot is None or r.owns_slot is False or snapshot_each_chunk:
            r.slot = cache.slot()
            r.owns_slot = True
        s_out.append(r.slot)
    kp = wp.kda_plan(num_heads=HK, head_dim_k=DK, head_dim_v=DK, num_state_slots=cache.state_pool.shape[0],
                     chunk_lens=chunk, state_in=s_in, state_out=s_out)
    kws = wp.new_workspace(kp, dev)
    kout = torch.empty((T, HK, DK), dtype=torch.bfloat16, device=dev)
    f32cat = lambda name: torch.cat([torch.as_tensor(getattr(reqs[ri], name)[s:s + l]) for ri, s, l in spans]).to(dev).contiguous()
    wp.kda_upload(kp, kws)
    wp.kda_chunked_prefill(kp, cat("kq"), cat("kk"), cat("kv"), f32cat("alpha"), f32cat("beta"), cache.state_pool,
                           kout, kws)
    torch.cuda.synchronize()
    o, ko = out.float().cpu().numpy(), kout.float().cpu().numpy()
    cu = 0
    for ri, s, l in spans:
        reqs[ri].out_attn[s:s + l] = o[cu:cu + l]
        reqs[ri].out_kda[s:s + l] = ko[cu:cu + l]
        cu += l
    return s_out


def oracle_check(r, lo):
    """Rows lo..n-1 of the request against the oracles over its whole prompt."""
    pos = np.arange(lo, r.n)
    G = HQ // HKV
    for h in range(HQ):
        o, _ = oracle.attention_rows(r.q[lo:, h].astype(np.float64), r.k[:, h // G].astype(np.float64),
                                     r.v[:, h // G].astype(np.float64), pos, SCALE)
        _compare.assert_parity(r.out_attn[lo:, h], o, what=f"attention head {h}")
    o_ref, _ = okda.kda_recurrence(np.zeros((HK, DK, DK)), r.kq.astype(np.float64), r.kk.astype(np.float64),
                                   r.kv.astype(np.float64), r.alpha.astype(np.float64), r.beta.astype(np.float64))
    _compare.assert_kda_parity(r.out_kda[lo:], o_ref[lo:], "kda")


def test_reuse_hints_planner_and_kernels_end_to_end():
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(2024)
    cache = Cache(num_pages=200, num_slots=32, dev=dev)
    A = Request(rng, 320)
    A.owns_slot = False
    # serve A cold in 128-token chunks; each chunk end leaves a snapshot in a slot of its own
    snapshots = {}                     # boundary (tokens) -> slot
    for start in range(0, A.n, 128):
        length = min(128, A.n - start)
        (slot,) = run_wave(cache, [A], [(0, start, length)], dev, snapshot_each_chunk=True)
        snapshots[start + length] = slot
    oracle_check(A, 0)
    assert sorted(snapshots) == [128, 256, 320]

    # hint index: A's blocks (window 0) and its snapshot boundaries (window 1)
    idx = wp.HintIndex(num_shards=8)
    _, a_keys = wp.block_hashes(A.tokens, B)
    idx.add(0, a_keys)
    idx.add(1, [a_keys[b // B - 1] for b in snapshots])

    # new requests sharing A's first 200 / 96 / 0 / 320 tokens
    news = [Request(rng, 450, A, 200), Request(rng, 300, A, 96), Request(rng, 257), Request(rng, 360, A, 320)]
    expect = [128, 0, 0, 320]          # attention endpoints 12 / 6 / 0 / 20 blocks, snapshots at 8, -, -, 20
    reqs = news
    planner = wp.MpuPlanner(max_budget=256, min_budget=64, block=B, stages=2, fills=1, max_lanes=8)
    starts = []
    for i, r in enumerate(reqs):
        _, keys = wp.block_hashes(r.tokens, B)
        att, probes = idx.probe_prefix(0, keys)
        rec, _ = idx.probe_recurrent(1, keys, att)
        reuse = rec * B
        assert reuse == expect[i], (i, att, rec)
        starts.append(reuse)
        if reuse:
            r.table = list(A.table[:reuse // B])         # share the cached pages
            r.slot = snapshots[reuse]                     # resume from the snapshot, do not overwrite it
        r.owns_slot = False
        planner.admit(i, reuse, r.n)

    waves = 0
    while True:
        spans, _ = planner.plan()
        if not spans:
            if planner.state()["ring"]:
                planner.retire()
                continue
            break
        planner.commit(spans)
        run_wave(cache, reqs, spans, dev)
        waves += 1
    assert waves >= 4
    for r, lo in zip(reqs, starts):
        assert not np.isnan(r.out_attn[lo:]).any() and not np.isnan(r.out_kda[lo:]).any()
        oracle_check(r, lo)
    # the reused snapshots were only read
    for b, slot in snapshots.items():
        assert all(r.slot != slot for r in reqs)


def test_mfma_probe_reports_a_plausible_rate_and_clock():
    """The measurement probe (wavepp_probe.h): its clock reading and its rate stay within what an
    MI355X can do (not a performance bar: a broken probe would read zero, negative or absurd)."""
    import ctypes
    lib = wp.load_library()
    lib.wavepp_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p]
    sink = torch.empty(256 * 512, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(4, dtype=torch.int64, device="cuda")
    s = torch.cuda.current_stream()
    assert lib.wavepp_probe_mfma(0, 10, 1, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(clocks.data_ptr()),
                                 ctypes.c_void_p(s.cuda_stream)) == -1
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(2):
        e0.record(s)
        assert lib.wavepp_probe_mfma(256, 2000, 1, ctypes.c_void_p(sink.data_ptr()),
                                     ctypes.c_void_p(clocks.data_ptr()), ctypes.c_void_p(s.cuda_stream)) == 0
        e1.record(s)
    torch.cuda.synchronize()
    c = clocks.cpu().numpy().astype(np.float64)
    ghz = (c[2] - c[0]) / ((c[3] - c[1]) * 10.0)
    tflops = 256 * 8 * 2000 * 4 * 32768.0 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    print(f"[probe] {tflops:.0f} TFLOP/s at {ghz:.2f} GHz", flush=True)
    assert 0.3 < ghz < 3.0
    assert 50.0 < tflops < 2600.0
    assert torch.isfinite(sink).all()


def test_hbm_read_probe_reads_every_word_once():
    """The read-bandwidth probe (wavepp_probe.h): every 32-bit word of the buffer is folded into the
    sink exactly once (the XOR of the sink equals the XOR of the buffer, including a ragged tail that
    is not a whole round of the grid), its argument checks reject bad sizes, and its rate stays below
    the HBM peak (not a performance bar)."""
    import ctypes
    lib = wp.load_library()
    lib.wavepp_probe_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_void_p]
    s = torch.cuda.current_stream()
    g = torch.Generator().manual_seed(77)
    for nbytes, wgs in ((16, 1), (1040, 3), (3 * (1 << 20) + 48, 37)):
        host = torch.randint(-(2 ** 31), 2 ** 31 - 1, (nbytes // 4,), dtype=torch.int64, generator=g).to(torch.int32)
        src = host.to("cuda")
        sink = torch.zeros(wgs * 256, dtype=torch.int32, device="cuda")
        assert lib.wavepp_probe_hbm_read(ctypes.c_void_p(src.data_ptr()), nbytes, wgs, ctypes.c_void_p(sink.data_ptr()),
                                         ctypes.c_void_p(s.cuda_stream)) == 0
        torch.cuda.synchronize()
        want = np.bitwise_xor.reduce(host.numpy().view(np.uint32))
        got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
        assert got == want, (nbytes, wgs)
    sink = torch.zeros(256, dtype=torch.int32, device="cuda")
    for nbytes, wgs in ((0, 1), (24, 1), (16, 0)):
        assert lib.wavepp_probe_hbm_read(ctypes.c_void_p(src.data_ptr()), nbytes, wgs, ctypes.c_void_p(sink.data_ptr()),
                                         ctypes.c_void_p(s.cuda_stream)) == -1
    import bench
    gbs = bench.hbm_read_probe(torch, mib=1024, workgroups=4096, launches=6)
    print(f"[read probe] {gbs:.0f} GB/s", flush=True)
    assert 500.0 < gbs < 8000.0
