"""Pins of the reuse-hint reference (CPU only).

* the hash primitive against the FIPS 180-2 example ("abc");
* chaining: a block's key depends on its whole prefix and nothing after it; equal prefixes give
  equal keys; salt and extra keys separate otherwise equal prefixes; only full blocks are hashed;
* the prefix endpoint through the index equals the longest common full-block prefix with the
  cached sequences, found by comparing tokens directly;
* counters: add / detach / erase at zero;
* the recurrent scan against brute force, and against the paper's worked example of recurrent
  endpoints diverging across two ranks (tests/golden/recurrent_fallback.json).
"""
import hashlib
import json
import os

import numpy as np
import pytest

from oracle import hints as oh

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_sha256_primitive_fips_example():
    assert hashlib.sha256(b"abc").hexdigest() == \
        "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"


def test_chaining_properties():
    rng = np.random.default_rng(0)
    B = 16
    toks = rng.integers(0, 1 << 20, 10 * B + 7).tolist()
    h = oh.chained_hashes(toks, B)
    assert len(h) == 10 and len(set(h)) == 10
    # a change in block 5 leaves blocks 0..4 and changes every key from 5 on
    t2 = list(toks)
    t2[5 * B + 3] += 1
    h2 = oh.chained_hashes(t2, B)
    assert h2[:5] == h[:5] and all(a != b for a, b in zip(h2[5:], h[5:]))
    # the partial tail block is not hashed and does not matter
    t3 = toks[:10 * B] + [1, 2, 3]
    assert oh.chained_hashes(t3, B) == h
    # the same block content after different prefixes gets different keys
    blockx = toks[:B]
    a = oh.chained_hashes(blockx + blockx, B)
    assert a[0] != a[1]
    # salt and extra keys
    assert oh.chained_hashes(toks, B, salt=b"tenant-1")[0] != h[0]
    extra = [None] * 10
    extra[3] = [7]
    he = oh.chained_hashes(toks, B, extra_keys=extra)
    assert he[:3] == h[:3] and all(x != y for x, y in zip(he[3:], h[3:]))


def test_counters():
    idx = oh.HintIndex()
    idx.add(0, [5, 6])
    idx.add(0, [5])
    idx.detach(0, [5])
    assert idx.contains(0, 5) and idx.contains(0, 6) and not idx.contains(1, 5)
    idx.detach(0, [5, 6])
    assert not idx.contains(0, 5) and not idx.contains(0, 6)
    with pytest.raises(KeyError):
        idx.detach(0, [5])


@pytest.mark.parametrize("seed", range(5))
def test_prefix_endpoint_equals_token_comparison(seed):
    rng = np.random.default_rng(seed)
    B = 8
    base = rng.integers(0, 50, 40 * B).tolist()
    cached = []
    idx = oh.HintIndex()
    for _ in range(6):                         # cached sequences share random prefixes of base
        cut = int(rng.integers(0, 40)) * B
        seq = base[:cut] + rng.integers(0, 50, int(rng.integers(0, 10)) * B).tolist()
        cached.append(seq)
        idx.add(3, [oh.key64(d) for d in oh.chained_hashes(seq, B)])
    for _ in range(10):
        cut = int(rng.integers(0, 40)) * B
        req = base[:cut] + rng.integers(0, 50, int(rng.integers(1, 80))).tolist()
        keys = [oh.key64(d) for d in oh.chained_hashes(req, B)]
        got = oh.prefix_endpoint(idx, 3, keys)
        want = 0
        for seq in cached:                     # longest common full-block prefix, token by token
            n = 0
            while (n + 1) * B <= min(len(seq), len(req)) and seq[n * B:(n + 1) * B] == req[n * B:(n + 1) * B]:
                n += 1
            want = max(want, n)
        assert got == want
        assert oh.prefix_endpoint(idx, 4, keys) == 0          # another window sees nothing


def test_recurrent_scan_brute_force():
    rng = np.random.default_rng(1)
    for _ in range(50):
        n = int(rng.integers(1, 30))
        keys = rng.integers(0, 1 << 60, n).tolist()
        snaps = oh.HintIndex()
        have = sorted(set(rng.integers(1, n + 1, int(rng.integers(0, 5))).tolist()))
        snaps.add(0, [keys[j - 1] for j in have])
        limit = int(rng.integers(0, n + 1))
        want = max([0] + [j for j in have if j <= limit])
        assert oh.recurrent_endpoint(snaps, 0, keys, limit) == want


def test_recurrent_fallback_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "recurrent_fallback.json")))
    blocks_per_k = 1024 // g["block"]
    n = 100 * blocks_per_k
    keys = list(range(1000, 1000 + n))
    ranks = []
    for snaps_k in g["rank_snapshots_k"]:
        idx = oh.HintIndex()
        idx.add(0, [keys[k * blocks_per_k - 1] for k in snaps_k])
        ranks.append(idx)
    for rank, start_k, end_k in g["steps"]:
        got = oh.recurrent_endpoint(ranks[rank], 0, keys, start_k * blocks_per_k)
        assert got == end_k * blocks_per_k
    # every rank can use the agreed endpoint
    for idx in ranks:
        a = g["agreed_k"] * blocks_per_k
        assert oh.recurrent_endpoint(idx, 0, keys, a) == a
