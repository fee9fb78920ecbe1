"""Host-side checks of libwavepp_attn.so that need no GPU: exports, validation, work list."""
import os
import re

import numpy as np
import pytest

import paper_2609_35263_amd as wp
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = wp.load_library()
    declared = set()
    for name in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if name.endswith(".h"):
            header = open(os.path.join(ROOT, "include", name)).read()
            declared |= set(re.findall(r"^(?:const\s+)?\w+\s*\*?\s*(wavepp_\w+)\s*\(", header, re.M))
    assert declared, "no declarations found"
    assert declared == (set(wp.EXPORTED_SYMBOLS) | set(wp.KDA_SYMBOLS) | set(wp.MPU_SYMBOLS) | set(wp.HINT_SYMBOLS)
                        | set(wp.PROBE_SYMBOLS))
    for name in declared:
        assert hasattr(lib, name), name


def kw(**over):
    base = dict(num_q_heads=8, num_kv_heads=2, head_dim_qk=64, head_dim_v=64, page_size=16, num_pages=16,
                softmax_scale=0.125, prefix_lens=[48], chunk_lens=[32], block_table=[[3, 7, 1, 12, 5, -1]])
    base.update(over)
    return base


def status_of(**over):
    try:
        wp.plan(**kw(**over))
        return 0
    except wp.WaveppError as e:
        return e.status


def test_valid_plan():
    p = wp.plan(**kw())
    info = p.info()
    assert info["total_tokens"] == 32 and info["num_real_items"] == 2   # 32 tokens x 4 heads = 128 rows, 2 kv heads
    assert p.workspace_bytes > 0 and p.workspace_bytes % 256 == 0


@pytest.mark.parametrize("over,status", [
    (dict(prefix_lens=[-1]), -1),
    (dict(chunk_lens=[-3]), -1),
    (dict(softmax_scale=0.0), -1),
    (dict(softmax_scale=float("inf")), -1),
    (dict(num_q_heads=6, num_kv_heads=4), -1),
    (dict(head_dim_qk=96, head_dim_v=96), -2),
    (dict(head_dim_qk=64, head_dim_v=128), -2),
    (dict(page_size=32), -2),
    (dict(kv_shared=True), -2),
    (dict(block_table=[[3, 7, 16, 12, 5, -1]]), -3),
    (dict(block_table=[[3, 7, 1, 12, -2, 0]]), -3),
    (dict(block_table=[[3, 7, 1, 12]]), -5),
    (dict(prefix_lens=[48, 0], chunk_lens=[32, 16], block_table=[[3, 7, 1, 12, 5], [5, 0, 0, 0, 0]]), -4),
    (dict(prefix_lens=[48, 16], chunk_lens=[32, 16], block_table=[[3, 7, 1, 12, 5], [12, 9, 0, 0, 0]]), -4),
    (dict(block_table=[[3, 7, 1, 5, 5, -1]]), -4),
])
def test_invalid_inputs_are_rejected(over, status):
    assert status_of(**over) == status


def test_shared_prefix_pages_and_ignored_entries_are_accepted():
    # two requests share prefix pages 3 and 7; entries past ceil(n/B) hold garbage
    assert status_of(prefix_lens=[32, 32], chunk_lens=[16, 20],
                     block_table=[[3, 7, 1, 10**6], [3, 7, 9, 11]]) == 0
    # an idle lane (c = 0) may share its pages freely
    assert status_of(prefix_lens=[48, 48], chunk_lens=[32, 0],
                     block_table=[[3, 7, 1, 12, 5], [3, 7, 1, 0, 0]]) == 0


def test_empty_and_idle_waves():
    p = wp.plan(**kw(prefix_lens=[], chunk_lens=[], block_table=np.zeros((0, 1), np.int32)))
    assert p.info()["num_items"] == 0
    p = wp.plan(**kw(prefix_lens=[10, 5], chunk_lens=[0, 0], block_table=[[1], [2]]))
    assert p.info()["num_items"] == 0 and p.info()["total_tokens"] == 0


def coverage_check(spec, items, kv_tile):
    """Each (request, kv head, row, key) visible pair is covered by exactly one work item."""
    G = spec.group_size
    seen = {}
    for (r, g, row0, rows, kb, ke, part, split) in items:
        if rows == 0:
            continue
        assert kb % kv_tile == 0 and ke > kb
        for row in range(row0, row0 + rows):
            seen.setdefault((r, g, row), []).append((kb, ke))
    for r in range(spec.num_requests):
        p, c = int(spec.prefix_lens[r]), int(spec.chunk_lens[r])
        for g in range(spec.num_kv_heads):
            for row in range(c * G):
                limit = p + row // G
                ranges = sorted(seen.pop((r, g, row)))
                # ranges partition [0, limit + 1) after clipping to the visible keys
                pos = 0
                for kb, ke in ranges:
                    assert kb == pos, (r, g, row, ranges)
                    pos = ke
                assert pos >= limit + 1, (r, g, row, ranges, limit)
    assert not seen


@pytest.mark.parametrize("splits", [0, 1, 2, 7])
def test_work_list_covers_every_visible_pair_once(splits):
    spec = wl.custom_wave(8, 2, 64, 64, 16, [48, 0, 5, 130], [32, 7, 0, 61], seed=4)
    p = wp.plan_for(spec, max_splits=splits)
    items = p.items()
    coverage_check(spec, items, p.info()["kv_tile"])
    info = p.info()
    assert info["max_splits"] <= max(splits, 1) or splits == 0
    parts = items[items[:, 6] >= 0]
    # partial rows of distinct splits never overlap
    spans = sorted((int(a), int(a) + int(b)) for a, b in zip(parts[:, 6], parts[:, 3]))
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    if spans:
        assert spans[-1][1] <= info["partial_rows"]


def test_work_list_cfg2_and_auto_splits():
    spec = wl.cfg2()
    p = wp.plan_for(spec)
    coverage_check(spec, p.items(), 64)
    small = wl.small_chunk(16)
    ps = wp.plan_for(small)
    assert ps.info()["max_splits"] > 1           # few rows, long prefixes: split to fill the chip
    coverage_check(small, ps.items(), 64)


def test_item_rows_follow_the_largest_chunk(monkeypatch):
    """128-row items (4-wave kernel form, two workgroups per CU) exactly when no (request, KV head)
    has more than 128 rows; WAVEPP_GQA_WAVES forces either form."""
    monkeypatch.delenv("WAVEPP_GQA_WAVES", raising=False)
    assert wp.plan_for(wl.small_chunk(16)).info()["rows_per_item"] == 128      # 16 tokens x G 8
    assert wp.plan_for(wl.small_chunk(32)).info()["rows_per_item"] == 256      # 32 x 8 = 256 rows
    assert wp.plan_for(wl.cfg1()).info()["rows_per_item"] == 128               # 32 x 4
    assert wp.plan_for(wl.cfg2()).info()["rows_per_item"] == 256
    edge = wl.custom_wave(16, 2, 64, 64, 16, [40, 3], [16, 15], seed=2)        # 16 x 8 = 128 rows: small
    assert wp.plan_for(edge).info()["rows_per_item"] == 128
    edge = wl.custom_wave(16, 2, 64, 64, 16, [40, 3], [17, 15], seed=2)        # 17 x 8 = 136 rows
    assert wp.plan_for(edge).info()["rows_per_item"] == 256
    monkeypatch.setenv("WAVEPP_GQA_WAVES", "8")
    assert wp.plan_for(wl.small_chunk(16)).info()["rows_per_item"] == 256
    monkeypatch.setenv("WAVEPP_GQA_WAVES", "4")
    p = wp.plan_for(wl.cfg2())
    assert p.info()["rows_per_item"] == 128
    coverage_check(wl.cfg2(), p.items(), p.info()["kv_tile"])


def test_kv_tile_is_the_kernel_form_tile(monkeypatch):
    """The 4-wave grouped form (128-row items) runs 64-key tiles and the 8-wave form 128-key tiles;
    the plan reports the tile of the form it chose and splits on whole tiles of it."""
    monkeypatch.delenv("WAVEPP_GQA_WAVES", raising=False)
    small = wl.small_chunk(16)
    ps = wp.plan_for(small)
    assert ps.info()["rows_per_item"] == 128 and ps.info()["kv_tile"] == 64
    coverage_check(small, ps.items(), 64)
    for splits in (3, 7):
        pf = wp.plan_for(small, max_splits=splits)
        coverage_check(small, pf.items(), 64)
        # forced splits cut at 64-key boundaries, so a split may start at an odd multiple of 64
        assert pf.info()["kv_tile"] == 64
    assert wp.plan_for(wl.cfg2()).info()["kv_tile"] == 128
    # automatic splits keep at least 1,024 keys each, in either form
    for spec in (small, wl.small_chunk(64), wl.cfg2()):
        items = wp.plan_for(spec).items()
        parts = items[(items[:, 6] >= 0) & (items[:, 3] > 0)]
        if len(parts):
            # every split but the last of its tile spans at least 1,024 keys
            for (r, g, row0, rows, kb, ke, part, split) in parts:
                later = parts[(parts[:, 0] == r) & (parts[:, 1] == g) & (parts[:, 2] == row0) & (parts[:, 7] > split)]
                if len(later):
                    assert ke - kb >= 1024, (r, g, row0, kb, ke)


def test_auto_splits_follow_request_length():
    """A wave split to fill the chip stays within 512 items, gives requests with longer prefixes at
    least as many splits as shorter ones, and keeps its items' key ranges within 20 % of their mean
    (the wave runs as one round of workgroups, so its longest item sets the interval)."""
    for c in (16, 32, 64):
        spec = wl.small_chunk(c)
        it = wp.plan_for(spec).items()
        real = it[it[:, 3] > 0]
        assert len(real) <= 512
        lens = real[:, 5] - real[:, 4]
        assert lens.max() <= 1.2 * lens.mean(), (c, lens.max(), lens.mean())
        splits = {}
        for r in real:
            splits[(int(r[0]), int(r[1]), int(r[2]))] = splits.get((int(r[0]), int(r[1]), int(r[2])), 0) + 1
        by_len = sorted((int(spec.prefix_lens[k[0]] + spec.chunk_lens[k[0]]), n) for k, n in splits.items())
        assert all(a[1] <= b[1] for a, b in zip(by_len, by_len[1:])), (c, by_len)
        coverage_check(spec, it, wp.plan_for(spec).info()["kv_tile"])


@pytest.mark.parametrize("seed", range(4))
def test_auto_splits_fuzz(seed):
    """Seeded random small waves with long prefixes, in both grouped forms and the latent one: the
    automatic splits cover every visible pair exactly once, keep the wave within 512 items, and cut
    no split but a range's last below the minimum split length."""
    rng = np.random.default_rng(900 + seed)
    for _ in range(6):
        Hq, Hkv, d, kv_shared = [(32, 8, 128, False), (16, 4, 64, False), (64, 8, 128, False),
                                 (16, 1, 576, True)][rng.integers(0, 4)]
        R = int(rng.integers(1, 9))
        G = Hq // Hkv
        max_c = max(1, (128 if kv_shared else 256) // G)
        prefix = (rng.integers(0, 9000, R) // 64) * 64 + rng.integers(0, 64, R) * (rng.random(R) < 0.5)
        chunk = rng.integers(1, max_c + 1, R)
        spec = wl.custom_wave(Hq, Hkv, d, 512 if kv_shared else d, 64, prefix, chunk, kv_shared=kv_shared,
                              seed=int(rng.integers(0, 1000)))
        p = wp.plan_for(spec)
        info, items = p.info(), p.items()
        coverage_check(spec, items, info["kv_tile"])
        real = items[items[:, 3] > 0]
        n_base = sum(-(-int(c) * G // info["rows_per_item"]) for c in chunk) * (1 if kv_shared else Hkv)
        if n_base < 512:
            assert len(real) <= 512, (len(real), n_base)
        min_keys = 512 if kv_shared else 1024
        parts = real[real[:, 6] >= 0]
        for (r, g, row0, rows, kb, ke, part, split) in parts:
            later = parts[(parts[:, 0] == r) & (parts[:, 1] == g) & (parts[:, 2] == row0) & (parts[:, 7] > split)]
            if len(later):
                assert ke - kb >= min_keys, (r, g, row0, kb, ke)


def test_plan_is_deterministic_and_independent_of_physical_pages():
    spec = wl.cfg2()
    a = wp.plan_for(spec).items()
    b = wp.plan_for(spec).items()
    assert np.array_equal(a, b)
    perm = np.random.default_rng(0).permutation(spec.num_pages).astype(np.int32)
    spec.block_table = perm[spec.block_table]
    c = wp.plan_for(spec).items()
    assert np.array_equal(a, c)


def test_latent_plan_shapes():
    ok = dict(num_q_heads=16, num_kv_heads=1, head_dim_qk=576, head_dim_v=512, page_size=64, num_pages=8,
              softmax_scale=1 / 24, prefix_lens=[100], chunk_lens=[30], block_table=[[1, 4, 0]], kv_shared=True)
    p = wp.plan(**ok)
    info = p.info()
    assert info["rows_per_item"] == 128 and info["kv_tile"] == 64 and info["num_real_items"] == 30 * 16 // 128 + 1
    for over, status in [(dict(num_kv_heads=2, num_q_heads=16), -2), (dict(head_dim_v=576), -2),
                         (dict(kv_shared=False), -2)]:
        try:
            wp.plan(**{**ok, **over})
            got = 0
        except wp.WaveppError as e:
            got = e.status
        assert got == status, (over, got)
    spec = wl.custom_wave(16, 1, 576, 512, 16, [37, 200, 5], [20, 1, 90], kv_shared=True, seed=1)
    for splits in (0, 2, 3):
        coverage_check(spec, wp.plan_for(spec, max_splits=splits).items(), 64)


def _fake_call_args(p):
    """Plausible-looking device addresses: these entry points must reject the call on the host,
    before they look at the buffers, so nothing is ever dereferenced."""
    return dict(ws=0x7f0000000000, ws_bytes=p.workspace_bytes + 4096)


def test_missing_or_stale_upload_is_an_error_before_any_launch():
    """append_kv and chunked_prefill refuse a workspace whose last upload was not this plan's (here:
    none at all), with WAVEPP_EINVAL and a message naming the upload call; no HIP call is made."""
    import ctypes
    lib = wp.load_library()
    p = wp.plan(**kw())
    a = _fake_call_args(p)
    vp = ctypes.c_void_p
    buf = vp(0x7f0000100000)
    st = lib.wavepp_attn_chunked_prefill(p.handle, buf, buf, buf, buf, None, vp(a["ws"]), a["ws_bytes"], None)
    assert st == -1
    assert b"wavepp_attn_plan_upload" in lib.wavepp_last_error()
    st = lib.wavepp_attn_append_kv(p.handle, buf, buf, buf, buf, vp(a["ws"]), a["ws_bytes"], None)
    assert st == -1
    assert b"wavepp_attn_plan_upload" in lib.wavepp_last_error()
    kp = wp.kda_plan(num_heads=2, head_dim_k=128, head_dim_v=128, num_state_slots=2, chunk_lens=[5],
                     state_in=[-1], state_out=[0])
    st = lib.wavepp_kda_chunked_prefill(kp.handle, buf, buf, buf, buf, buf, buf, buf, vp(a["ws"]),
                                        kp.workspace_bytes + 4096, None)
    assert st == -1
    assert b"wavepp_kda_upload" in lib.wavepp_last_error()


def test_binding_rejects_tensors_whose_shape_does_not_match_the_plan():
    torch = pytest.importorskip("torch")
    bf = torch.bfloat16
    p = wp.plan(**kw())          # T = 32, Hq 8, Hkv 2, d 64, B 16, P 16
    ws = torch.empty(p.workspace_bytes, dtype=torch.uint8)
    good = dict(q=torch.empty(32, 8, 64, dtype=bf), k_pool=torch.empty(16, 2, 16, 64, dtype=bf),
                v_pool=torch.empty(16, 2, 16, 64, dtype=bf), out=torch.empty(32, 8, 64, dtype=bf),
                lse=torch.empty(32, 8, dtype=torch.float32))
    bad = dict(q=torch.empty(31, 8, 64, dtype=bf), k_pool=torch.empty(15, 2, 16, 64, dtype=bf),
               v_pool=torch.empty(16, 2, 16, 32, dtype=bf), out=torch.empty(32, 8, 32, dtype=bf),
               lse=torch.empty(32, 4, dtype=torch.float32))
    for name in good:
        args = dict(good)
        args[name] = bad[name]
        with pytest.raises(ValueError, match="shape"):
            wp.chunked_prefill(p, args["q"], args["k_pool"], args["v_pool"], args["out"], args["lse"], ws)
    kn = torch.empty(32, 2, 64, dtype=bf)
    with pytest.raises(ValueError, match="shape"):
        wp.append_kv(p, kn[:31], kn, good["k_pool"], good["v_pool"], ws)
    with pytest.raises(ValueError, match="shape"):
        wp.append_kv(p, kn, kn, good["k_pool"], torch.empty(16, 2, 8, 64, dtype=bf), ws)
    with pytest.raises(ValueError, match="required"):
        wp.append_kv(p, kn, None, good["k_pool"], good["v_pool"], ws)
    # right shapes, host memory: rejected as not on the device
    with pytest.raises(ValueError, match="device"):
        wp.chunked_prefill(p, good["q"], good["k_pool"], good["v_pool"], good["out"], good["lse"], ws)
    kp = wp.kda_plan(num_heads=2, head_dim_k=128, head_dim_v=128, num_state_slots=3, chunk_lens=[5, 2],
                     state_in=[-1, 0], state_out=[1, 2])
    f32 = torch.float32
    kgood = dict(q=torch.empty(7, 2, 128, dtype=bf), k=torch.empty(7, 2, 128, dtype=bf),
                 v=torch.empty(7, 2, 128, dtype=bf), alpha=torch.empty(7, 2, 128, dtype=f32),
                 beta=torch.empty(7, 2, dtype=f32), state_pool=torch.empty(3, 2, 128, 128, dtype=f32),
                 out=torch.empty(7, 2, 128, dtype=bf))
    for name, t in kgood.items():
        args = dict(kgood)
        args[name] = t[:-1]
        with pytest.raises(ValueError, match="shape"):
            wp.kda_chunked_prefill(kp, args["q"], args["k"], args["v"], args["alpha"], args["beta"],
                                   args["state_pool"], args["out"], ws)


def _expected_status(Hq, Hkv, dq, dv, B, P, kv_shared, prefix, chunk, bt):
    """The validation rules of the plan, restated: shape, then each request in order (lengths,
    span backed by the table, entries inside the pool), then pages receiving appended tokens must
    be referenced exactly once among all entries that are read."""
    if Hq % Hkv:
        return -1
    ok_dims = ((dq, dv) == (576, 512) and Hkv == 1) if kv_shared else (dq, dv) in ((64, 64), (128, 128))
    if B not in (16, 64) or not ok_dims:
        return -2
    ref = np.zeros(P, np.int64)
    for r in range(len(prefix)):
        p, c = int(prefix[r]), int(chunk[r])
        if p < 0 or c < 0:
            return -1
        if p + c > bt.shape[1] * B:
            return -5
        for b in range(-(-(p + c) // B)):
            if not 0 <= bt[r, b] < P:
                return -3
            ref[bt[r, b]] += 1
    for r in range(len(prefix)):
        p, c = int(prefix[r]), int(chunk[r])
        if c and any(ref[bt[r, b]] != 1 for b in range(p // B, -(-(p + c) // B))):
            return -4
    return 0


@pytest.mark.parametrize("seed", range(6))
def test_plan_fuzz_against_restated_rules(seed):
    """Seeded random waves: random spans, shared / aliased / out-of-range / short block tables, head
    shapes and forced splits.  The status must be the restated rules' status, and every accepted
    plan's work list must cover every visible pair exactly once."""
    rng = np.random.default_rng(100 + seed)
    seen = set()
    for _ in range(60):
        shape = [(8, 2, 64, 64, False), (16, 4, 128, 128, False), (16, 1, 576, 512, True), (6, 4, 64, 64, False),
                 (8, 2, 96, 96, False), (8, 1, 576, 512, False)][rng.integers(0, 6)]
        Hq, Hkv, dq, dv, kv_shared = shape
        B = int(rng.choice([16, 64, 16, 64, 32]))
        P = int(rng.integers(1, 40))
        R = int(rng.integers(0, 5))
        stride = int(rng.integers(1, 9))
        prefix = rng.integers(0, 150, R)
        chunk = rng.integers(0, 120, R) * (rng.random(R) > 0.15)
        if R and rng.random() < 0.05:
            prefix[rng.integers(0, R)] = -1
        if rng.random() < 0.6:
            bt = np.resize(rng.permutation(P), (max(R, 1), stride)).astype(np.int32)[:R]
        else:
            bt = rng.integers(0, P, (R, stride)).astype(np.int32)
        if R > 1 and rng.random() < 0.3:
            bt[1, 0] = bt[0, 0]                      # a shared first page
        if R and rng.random() < 0.1:
            bt[rng.integers(0, R), rng.integers(0, stride)] = int(rng.choice([-1, P]))
        bt = bt.reshape(R, stride)
        want = _expected_status(Hq, Hkv, dq, dv, B, P, kv_shared, prefix, chunk, bt)
        splits = int(rng.choice([0, 0, 1, 2, 5]))
        try:
            p = wp.plan(num_q_heads=Hq, num_kv_heads=Hkv, head_dim_qk=dq, head_dim_v=dv, page_size=B, num_pages=P,
                        softmax_scale=0.1, prefix_lens=prefix, chunk_lens=chunk,
                        block_table=bt if R else np.zeros((0, stride), np.int32), kv_shared=kv_shared,
                        max_splits=splits)
            got = 0
        except wp.WaveppError as e:
            got = e.status
        assert got == want, (shape, B, P, prefix, chunk, bt)
        seen.add(got)
        if got == 0:
            spec = wl.custom_wave(Hq, Hkv, dq, dv, B, prefix, chunk, kv_shared=kv_shared, num_pages=P, seed=1)
            spec.block_table = bt
            coverage_check(spec, p.items(), p.info()["kv_tile"])
    assert 0 in seen


def test_noalloc_entry_point_rejects_plans_beyond_its_static_scratch():
    """The allocation-free entry point checks the plan's scratch need against its fixed 160 MiB array
    before any HIP call."""
    import ctypes
    lib = wp.load_library()
    spec = wl.small_chunk(128)
    p = wp.plan_for(spec, max_splits=64)
    assert p.workspace_bytes > 160 << 20
    vp = ctypes.c_void_p
    buf = vp(0x7f0000100000)
    st = lib.wavepp_attn_chunked_prefill_noalloc(p.handle, buf, None, None, buf, buf, buf, None, None)
    assert st == -6
    assert b"static scratch" in lib.wavepp_last_error()
    # a plan that fits passes the size check (and then needs a GPU: not called here)
    assert wp.plan_for(spec).workspace_bytes <= 160 << 20
