"""The native reuse-hint machinery (C ABI) against the reference (CPU only): bit-exact chained
hashes, the counted index under random add / detach, probe endpoints, the O(log N) probe bound,
and concurrent use from several threads."""
import math
import threading

import numpy as np
import pytest

import paper_2609_35263_amd as wp
from oracle import hints as oh


@pytest.mark.parametrize("block,extra,salt_len", [(1, 0, 19), (1, 0, 20), (1, 0, 27), (1, 0, 28), (1, 0, 83),
                                                  (1, 0, 84), (16, 0, 0), (64, 0, 5), (63, 2, 0), (64, 3, 31),
                                                  (5, 1, 64)])
def test_hashes_bit_exact(block, extra, salt_len):
    """Message lengths 36 + salt_len cover SHA-256's padding edges (55, 56, 63, 64, 119, 120 bytes)."""
    rng = np.random.default_rng(block * 100 + extra * 10 + salt_len)
    toks = rng.integers(-(1 << 31), 1 << 31, 7 * block + min(3, block - 1), dtype=np.int64).astype(np.int32)
    salt = bytes(rng.integers(0, 256, salt_len, dtype=np.int64).astype(np.uint8))
    ek = rng.integers(-(1 << 62), 1 << 62, (7, extra), dtype=np.int64) if extra else None
    dig, keys = wp.block_hashes(toks, block, ek, salt)
    ref = oh.chained_hashes(toks.tolist(), block, None if ek is None else ek.tolist(), salt)
    assert len(dig) == len(ref) == 7
    for i in range(7):
        assert bytes(dig[i]) == ref[i]
        assert int(keys[i]) == oh.key64(ref[i])


def test_index_counts_match_reference():
    rng = np.random.default_rng(3)
    nat, ref = wp.HintIndex(num_shards=7), oh.HintIndex()
    pool = rng.integers(0, 1 << 63, 200, dtype=np.int64).astype(np.uint64)
    for _ in range(2000):
        w = int(rng.integers(0, 3))
        ks = pool[rng.integers(0, 200, int(rng.integers(1, 5)))]
        if rng.random() < 0.6:
            nat.add(w, ks)
            ref.add(w, [int(x) for x in ks])
        else:
            ks = [k for k in ks if ref.contains(w, int(k))][:1]
            if ks:
                nat.detach(w, ks)
                ref.detach(w, [int(x) for x in ks])
    assert nat.size() == len(ref.count)
    for w in range(3):
        for k in pool:
            assert (nat.probe_prefix(w, [k])[0] == 1) == ref.contains(w, int(k))
    with pytest.raises(wp.WaveppError):
        nat.detach(9, [1])


@pytest.mark.parametrize("seed", range(6))
def test_prefix_probe_matches_plain_scan_on_cache_trees(seed):
    rng = np.random.default_rng(seed)
    B = 16
    base = rng.integers(0, 1000, 300 * B)
    nat, ref = wp.HintIndex(), oh.HintIndex()
    for _ in range(8):                           # cached sequences: prefixes of base plus private blocks
        cut = int(rng.integers(0, 300)) * B
        seq = np.concatenate([base[:cut], rng.integers(0, 1000, int(rng.integers(0, 20)) * B)])
        _, keys = wp.block_hashes(seq, B)
        nat.add(0, keys)
        ref.add(0, [int(k) for k in keys])
    for _ in range(30):
        cut = int(rng.integers(0, 300)) * B
        req = np.concatenate([base[:cut], rng.integers(0, 1000, int(rng.integers(0, 40 * B)))])
        _, keys = wp.block_hashes(req, B)
        want = oh.prefix_endpoint(ref, 0, [int(k) for k in keys])
        got, probes = nat.probe_prefix(0, keys)
        lin, lin_probes = nat.probe_prefix_linear(0, keys)
        assert got == want == lin
        n = len(keys)
        assert probes <= 2 * math.ceil(math.log2(n + 1)) + 1
        assert lin_probes == min(n, want + 1)


def test_prefix_probe_result_is_a_boundary_on_any_set():
    """Off trees (a stale or concurrently changing view) the probe still returns a hit / miss boundary."""
    rng = np.random.default_rng(11)
    for _ in range(200):
        n = int(rng.integers(0, 60))
        keys = rng.integers(1, 1 << 62, n, dtype=np.int64).astype(np.uint64)
        present = rng.random(n) < 0.7
        nat = wp.HintIndex(num_shards=3)
        nat.add(1, keys[present])
        e, _ = nat.probe_prefix(1, keys)
        assert 0 <= e <= n
        assert e == 0 or present[e - 1]
        assert e == n or not present[e]


def test_recurrent_probe_matches_reference():
    rng = np.random.default_rng(12)
    for _ in range(100):
        n = int(rng.integers(1, 80))
        keys = rng.integers(1, 1 << 62, n, dtype=np.int64).astype(np.uint64)
        snaps = keys[rng.random(n) < 0.1]
        nat, ref = wp.HintIndex(), oh.HintIndex()
        nat.add(2, snaps)
        ref.add(2, [int(k) for k in snaps])
        limit = int(rng.integers(0, n + 1))
        got, probes = nat.probe_recurrent(2, keys, limit)
        assert got == oh.recurrent_endpoint(ref, 2, [int(k) for k in keys], limit)
        assert probes == (limit - got + 1 if got > 0 else limit)


def test_concurrent_updates_and_probes():
    B, n_threads = 16, 6
    rng = np.random.default_rng(13)
    seqs = [rng.integers(0, 1000, 200 * B) for _ in range(n_threads)]
    keysets = [wp.block_hashes(s, B)[1] for s in seqs]
    idx = wp.HintIndex(num_shards=16)
    errors = []

    def writer(i):
        try:
            for _ in range(20):
                idx.add(0, keysets[i])
                idx.detach(0, keysets[i])
            idx.add(0, keysets[i])
        except Exception as e:        # noqa: BLE001
            errors.append(e)

    def reader(i):
        try:
            for _ in range(200):
                e, _ = idx.probe_prefix(0, keysets[i])
                assert 0 <= e <= len(keysets[i])
        except Exception as e:        # noqa: BLE001
            errors.append(e)

    th = [threading.Thread(target=writer, args=(i,)) for i in range(n_threads)] + \
         [threading.Thread(target=reader, args=(i,)) for i in range(n_threads)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not errors
    assert idx.size() == sum(len(set(k.tolist())) for k in keysets)
    for k in keysets:
        assert idx.probe_prefix(0, k)[0] == len(k)
