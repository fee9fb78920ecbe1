"""Structure of the seeded synthetic waves (CPU only)."""
import numpy as np
import pytest

import workloads as wl


def test_cfg1_shape_and_pairs():
    s = wl.cfg1()
    assert (s.num_q_heads, s.num_kv_heads, s.head_dim_qk, s.page_size, s.num_pages) == (8, 2, 64, 16, 16)
    assert list(s.prefix_lens) == [48] and list(s.chunk_lens) == [32]
    assert s.softmax_scale == 1 / 8
    # 48 * 32 + 32 * 33 / 2 visible pairs per head
    assert int(s.pairs().sum()) == 2064
    assert len(set(s.block_table[0, :5].tolist())) == 5


def test_budget_ladder_halves_to_floor():
    # Eq. 6 with the matched PP4 setting M = 16384, b_min = 8192, and the chunk ladder of cfg3
    assert wl.budget_ladder(16384, 8192, 64) == [16384, 8192]
    assert wl.budget_ladder(4096, 512, 64) == [4096, 2048, 1024, 512]
    assert wl.budget_ladder(1000, 100, 64) == [1000, 448, 192, 100]


def test_cfg2_structure():
    s = wl.cfg2()
    assert s.num_pages == 512 and s.num_requests == 4
    assert np.all(s.prefix_lens % 64 == 0) and np.all(s.prefix_lens <= 4096)
    assert np.all(s.chunk_lens == 2048)
    used = np.concatenate([s.block_table[r, :wl.ceil_div(int(s.prefix_lens[r] + 2048), 64)] for r in range(4)])
    assert len(set(used.tolist())) == len(used)
    assert used.min() >= 0 and used.max() < 512


def test_cfg3_shared_prefix():
    s = wl.cfg3()
    assert s.num_requests == 32
    assert all(np.array_equal(s.block_table[0, :256], s.block_table[r, :256]) for r in range(32))
    assert set(s.chunk_lens.tolist()) <= {4096, 2048, 1024, 512}
    assert np.all((s.prefix_lens - 16384) % 64 == 0) and np.all(s.prefix_lens - 16384 <= 2048)
    cnt = wl.prefix_slot_counts(s)
    assert np.all(cnt[s.block_table[0, :256]] == 64)


def test_cfg4_budget_split():
    s = wl.cfg4()
    assert s.layers == 4
    assert s.total_tokens <= 16384 and 16384 - s.total_tokens < 128
    assert np.all(s.chunk_lens >= 128) and np.all(s.chunk_lens <= 4096)
    assert 4 <= s.num_requests <= 16
    assert np.any(s.prefix_lens % 64 != 0)          # mid-page starts


def test_cfg5_and_6p_shapes():
    s = wl.cfg5()
    assert s.kv_shared and (s.head_dim_qk, s.head_dim_v, s.num_kv_heads, s.num_q_heads) == (576, 512, 1, 128)
    assert s.num_pages == 17408 and s.total_tokens == 65536
    s6 = wl.cfg6p()
    assert np.all(s6.prefix_lens == 124992) and np.all(s6.chunk_lens == 4096)


def test_tensors_poison_only_uncached_slots():
    s = wl.custom_wave(4, 2, 8, 8, 4, [5, 0, 9], [6, 3, 2], seed=1)
    t = wl.make_tensors(s, seed=3, poison=True)
    k = t["k_pool"].float().numpy()
    cnt = wl.prefix_slot_counts(s)
    for page in range(s.num_pages):
        for slot in range(4):
            assert np.isnan(k[page, :, slot]).all() == (slot >= cnt[page])
    t0 = wl.make_tensors(s, seed=3, poison=False)
    assert np.isfinite(t0["k_pool"].float().numpy()).all()
    t1 = wl.make_tensors(s, seed=3, poison=True)
    assert np.array_equal(wl.to_bits(t1["q"]), wl.to_bits(t["q"]))
