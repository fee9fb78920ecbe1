"""Pins of the fp64 oracle against things other than itself (CPU only).

* library cross-check: torch's scaled_dot_product_attention (fp64, causal, GQA) over the
  contiguous sequence, last c rows;
* closed forms from tests/golden/closed_forms.json and brute force at 1-4 tokens;
* invariants: chunking, page permutation, GQA = expanded MHA, latent = generic, row sums,
  split-and-merge, needles;
* the append: round trip, untouched slots, brute-force slot scan;
* teeth: the parity harness rejects the oracle with a page dropped, a page mis-mapped or the
  causal diagonal shifted.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import attention as oa
import workloads as wl
from tests import _compare

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
NAN = wl.BF16_NAN_BITS


def f32_to_bf16_bits(x):
    return wl.to_bits(torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16))


def rand_bits(rng, shape, scale=1.0):
    return f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * scale)


class Seq:
    """A wave built from contiguous per-request sequences, scattered into a permuted page pool by
    explicit position loops (independent of the oracle's gather)."""

    def __init__(self, Hq, Hkv, d, B, prefix, chunk, seed=0, dv=None, extra_pages=3, bt_fill=-1):
        rng = np.random.default_rng(seed)
        dv = d if dv is None else dv
        self.Hq, self.Hkv, self.d, self.dv, self.B = Hq, Hkv, d, dv, B
        self.prefix = np.asarray(prefix, np.int32)
        self.chunk = np.asarray(chunk, np.int32)
        n = self.prefix + self.chunk
        nb = [-(-int(x) // B) for x in n]
        self.P = sum(nb) + extra_pages
        perm = rng.permutation(self.P)
        self.bt = np.full((len(n), max(nb + [1]) + 2), bt_fill, np.int32)
        cur = 0
        for r, k in enumerate(nb):
            self.bt[r, :k] = perm[cur:cur + k]
            cur += k
        self.kseq = [rand_bits(rng, (int(x), Hkv, d)) for x in n]
        self.vseq = [rand_bits(rng, (int(x), Hkv, dv)) for x in n]
        self.qseq = [rand_bits(rng, (int(x), Hq, d)) for x in n]
        self.k_pool = np.full((self.P, Hkv, B, d), NAN, np.uint16)
        self.v_pool = np.full((self.P, Hkv, B, dv), NAN, np.uint16)
        for r in range(len(n)):
            for j in range(int(n[r])):
                page, slot = self.bt[r, j // B], j % B
                self.k_pool[page, :, slot, :] = self.kseq[r][j]
                self.v_pool[page, :, slot, :] = self.vseq[r][j]
        self.q = np.concatenate([self.qseq[r][int(self.prefix[r]):] for r in range(len(n))], axis=0)

    def run(self, scale=None, **kw):
        scale = 1.0 / math.sqrt(self.d) if scale is None else scale
        return oracle.chunked_prefill(self.q, self.k_pool, self.v_pool, self.prefix, self.chunk, self.bt,
                                      page_size=self.B, num_kv_heads=self.Hkv, softmax_scale=scale, **kw)


def sdpa_reference(seq, scale):
    outs = []
    for r in range(len(seq.prefix)):
        p, c = int(seq.prefix[r]), int(seq.chunk[r])
        if c == 0:
            continue
        q = torch.from_numpy(oracle.bf16_bits_to_f64(seq.qseq[r])).permute(1, 0, 2)[None]
        k = torch.from_numpy(oracle.bf16_bits_to_f64(seq.kseq[r])).permute(1, 0, 2)[None]
        v = torch.from_numpy(oracle.bf16_bits_to_f64(seq.vseq[r])).permute(1, 0, 2)[None]
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True, scale=scale,
                                                             enable_gqa=True)
        outs.append(o[0].permute(1, 0, 2)[p:p + c].numpy())
    return np.concatenate(outs, axis=0)


CASES = [
    # Hq, Hkv, d, B, prefix, chunk
    (4, 2, 8, 4, [0, 5, 12], [7, 1, 9]),
    (8, 2, 16, 16, [48], [32]),
    (6, 3, 4, 1, [3, 0], [2, 4]),
    (2, 1, 32, 2, [7, 3], [0, 5]),
    (8, 8, 16, 4, [9, 4], [3, 5]),
    (4, 1, 16, 8, [17], [6]),
    (4, 2, 8, 16, [35, 64, 1], [29, 16, 70]),
]


@pytest.mark.parametrize("case", CASES)
def test_sdpa_crosscheck(case):
    Hq, Hkv, d, B, prefix, chunk = case
    seq = Seq(Hq, Hkv, d, B, prefix, chunk, seed=len(prefix) * 7 + d)
    scale = 1.0 / math.sqrt(d)
    o, lse = seq.run(scale)
    ref = sdpa_reference(seq, scale)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    assert np.max(np.abs(o - ref)) <= 1e-12


def test_identity_table_equals_contiguous():
    # With Hkv = 1 and block table = arange, the pool reshaped [P*B, d] is the sequence itself.
    rng = np.random.default_rng(5)
    B, P, d = 4, 5, 8
    k_pool = rand_bits(rng, (P, 1, B, d))
    v_pool = rand_bits(rng, (P, 1, B, d))
    p, c = 13, 7
    q = rand_bits(rng, (c, 2, d))
    bt = np.arange(P, dtype=np.int32)[None]
    o, _ = oracle.chunked_prefill(q, k_pool, v_pool, [p], [c], bt, page_size=B, num_kv_heads=1,
                                  softmax_scale=0.3)
    kseq = torch.from_numpy(oracle.bf16_bits_to_f64(k_pool.reshape(P * B, d)[:p + c]))
    vseq = torch.from_numpy(oracle.bf16_bits_to_f64(v_pool.reshape(P * B, d)[:p + c]))
    qf = torch.from_numpy(oracle.bf16_bits_to_f64(q))
    for h in range(2):
        mask = torch.arange(p + c)[None, :] <= (p + torch.arange(c))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(qf[:, h][None], kseq[None], vseq[None],
                                                               attn_mask=mask[None], scale=0.3)[0]
        assert np.max(np.abs(o[:, h] - ref.numpy())) <= 1e-12


@pytest.mark.parametrize("name", ["two_keys", "three_keys_mean", "two_keys_scaled"])
def test_golden_closed_forms(name):
    case = json.load(open(os.path.join(GOLDEN, "closed_forms.json")))[name]
    B, p, c = case["page_size"], case["prefix_len"], case["chunk_len"]
    n = p + c
    P = -(-n // B) + 1
    bt = np.arange(P, dtype=np.int32)[::-1].copy()[None]      # reversed physical order
    k_pool = np.full((P, 1, B, 1), NAN, np.uint16)
    v_pool = np.full((P, 1, B, 1), NAN, np.uint16)
    kb, vb = f32_to_bf16_bits(case["k"]), f32_to_bf16_bits(case["v"])
    for j in range(n):
        k_pool[bt[0, j // B], 0, j % B, 0] = kb[j]
        v_pool[bt[0, j // B], 0, j % B, 0] = vb[j]
    q = f32_to_bf16_bits(case["q"]).reshape(c, 1, 1)
    o, lse = oracle.chunked_prefill(q, k_pool, v_pool, [p], [c], bt, page_size=B, num_kv_heads=1,
                                    softmax_scale=case["scale"])
    assert abs(o[-1, 0, 0] - case["o"]) <= 1e-14
    assert abs(lse[-1, 0] - case["lse"]) <= 1e-14


def test_single_visible_key_is_exact():
    seq = Seq(4, 2, 8, 4, [0], [1], seed=3)
    o, lse = seq.run(0.7)
    v0 = oracle.bf16_bits_to_f64(seq.vseq[0][0])        # [Hkv, d]
    for h in range(4):
        assert np.array_equal(o[0, h], v0[h // 2])
    s = 0.7 * np.einsum("hd,hd->h", oracle.bf16_bits_to_f64(seq.q[0]),
                        np.repeat(oracle.bf16_bits_to_f64(seq.kseq[0][0]), 2, axis=0))
    assert np.max(np.abs(lse[0] - s)) <= 1e-14


def test_zero_query_and_identical_keys_give_mean():
    seq = Seq(2, 1, 8, 2, [3], [3], seed=4)
    seq.q[:] = 0
    o, lse = seq.run(1.0)
    v = oracle.bf16_bits_to_f64(seq.vseq[0][:, 0])
    for i in range(3):
        np.testing.assert_allclose(o[i, 0], v[:3 + i + 1].mean(axis=0), rtol=0, atol=1e-14)
        assert abs(lse[i, 0] - math.log(3 + i + 1)) <= 1e-14
    # identical keys: every visible logit is equal whatever q is
    seq2 = Seq(2, 1, 8, 2, [3], [3], seed=5)
    for r in range(1):
        for j in range(6):
            seq2.k_pool[seq2.bt[r, j // 2], :, j % 2, :] = seq2.kseq[r][0]
    o2, _ = seq2.run(1.0)
    v2 = oracle.bf16_bits_to_f64(seq2.vseq[0][:, 0])
    for i in range(3):
        np.testing.assert_allclose(o2[i, 0], v2[:3 + i + 1].mean(axis=0), rtol=0, atol=1e-13)


def brute_force(seq, scale):
    """Scalar loops: look up each visible position's page by hand and sum exponentials."""
    res = []
    cu = 0
    G = seq.Hq // seq.Hkv
    for r in range(len(seq.prefix)):
        p, c = int(seq.prefix[r]), int(seq.chunk[r])
        for i in range(c):
            row = []
            for h in range(seq.Hq):
                qv = [float(x) for x in oracle.bf16_bits_to_f64(seq.q[cu + i, h])]
                logits, vals = [], []
                for j in range(p + i + 1):
                    page, slot = int(seq.bt[r, j // seq.B]), j % seq.B
                    kv = oracle.bf16_bits_to_f64(seq.k_pool[page, h // G, slot])
                    vv = oracle.bf16_bits_to_f64(seq.v_pool[page, h // G, slot])
                    logits.append(scale * math.fsum(a * b for a, b in zip(qv, kv)))
                    vals.append(vv)
                mx = max(logits)
                w = [math.exp(s - mx) for s in logits]
                tot = math.fsum(w)
                row.append(sum(wj * vj for wj, vj in zip(w, vals)) / tot)
            res.append(row)
        cu += c
    return np.asarray(res)


@pytest.mark.parametrize("B", [1, 2, 4])
def test_brute_force_tiny(B):
    for n in range(1, 5):
        for c in range(1, n + 1):
            p = n - c
            seq = Seq(4, 2, 3, B, [p], [c], seed=100 * B + 10 * n + c)
            o, _ = seq.run(0.9)
            bf = brute_force(seq, 0.9)
            assert np.max(np.abs(o - bf)) <= 1e-12, (B, p, c)


def test_row_sums_and_causal_zeros():
    seq = Seq(4, 2, 8, 4, [5, 0], [6, 3], seed=8)
    for r in range(2):
        for h in range(4):
            P = oracle.probabilities(seq.q, seq.k_pool, seq.prefix, seq.chunk, seq.bt, r, h, page_size=4,
                                     num_kv_heads=2, softmax_scale=0.5)
            p, c = int(seq.prefix[r]), int(seq.chunk[r])
            assert P.shape == (c, p + c)
            assert np.max(np.abs(P.sum(axis=1) - 1.0)) <= 1e-12
            for i in range(c):
                assert np.all(P[i, p + i + 1:] == 0.0)
                assert np.all(P[i, :p + i + 1] > 0.0)


def test_chunking_invariance():
    Hq, Hkv, d, B = 4, 2, 8, 4
    rng = np.random.default_rng(11)
    p, total = 9, 17
    chunks = [5, 1, 11]
    n = p + total
    P = -(-n // B) + 4
    bt = rng.permutation(P)[: -(-n // B)].astype(np.int32)[None]
    k_pool = np.full((P, Hkv, B, d), NAN, np.uint16)
    v_pool = np.full((P, Hkv, B, d), NAN, np.uint16)
    kp, vp = rand_bits(rng, (p, Hkv, d)), rand_bits(rng, (p, Hkv, d))
    for j in range(p):
        k_pool[bt[0, j // B], :, j % B] = kp[j]
        v_pool[bt[0, j // B], :, j % B] = vp[j]
    k_new, v_new, q = rand_bits(rng, (total, Hkv, d)), rand_bits(rng, (total, Hkv, d)), rand_bits(rng, (total, Hq, d))
    kw = dict(page_size=B, num_kv_heads=Hkv, softmax_scale=0.4)
    k1, v1 = oracle.append_kv(k_pool, v_pool, k_new, v_new, [p], [total], bt, B)
    o_full, l_full = oracle.chunked_prefill(q, k1, v1, [p], [total], bt, **kw)
    kc, vc = k_pool, v_pool
    start, outs, lses = p, [], []
    off = 0
    for c in chunks:
        kc, vc = oracle.append_kv(kc, vc, k_new[off:off + c], v_new[off:off + c], [start], [c], bt, B)
        o, l = oracle.chunked_prefill(q[off:off + c], kc, vc, [start], [c], bt, **kw)
        outs.append(o)
        lses.append(l)
        start += c
        off += c
    assert np.max(np.abs(np.concatenate(outs) - o_full)) <= 1e-12
    assert np.max(np.abs(np.concatenate(lses) - l_full)) <= 1e-12
    assert np.array_equal(kc, k1) and np.array_equal(vc, v1)


def test_page_permutation_invariance():
    seq = Seq(4, 2, 8, 4, [10, 3], [6, 9], seed=21, extra_pages=5)
    o, lse = seq.run(0.5)
    perm = np.random.default_rng(2).permutation(seq.P)
    kp = np.empty_like(seq.k_pool)
    vp = np.empty_like(seq.v_pool)
    kp[perm] = seq.k_pool
    vp[perm] = seq.v_pool
    bt = np.where(seq.bt >= 0, perm[np.maximum(seq.bt, 0)], -1).astype(np.int32)
    o2, lse2 = oracle.chunked_prefill(seq.q, kp, vp, seq.prefix, seq.chunk, bt, page_size=4, num_kv_heads=2,
                                      softmax_scale=0.5)
    assert np.array_equal(o, o2) and np.array_equal(lse, lse2)


def test_gqa_equals_expanded_mha():
    seq = Seq(8, 2, 8, 4, [7, 2], [5, 6], seed=31)
    o, lse = seq.run(0.3)
    G = 4
    k_exp = np.repeat(seq.k_pool, G, axis=1)
    v_exp = np.repeat(seq.v_pool, G, axis=1)
    o2, lse2 = oracle.chunked_prefill(seq.q, k_exp, v_exp, seq.prefix, seq.chunk, seq.bt, page_size=4,
                                      num_kv_heads=8, softmax_scale=0.3)
    assert np.array_equal(o, o2) and np.array_equal(lse, lse2)


def test_latent_equals_generic():
    seq = Seq(6, 1, 24, 4, [9, 0], [4, 7], seed=41)
    o, lse = oracle.chunked_prefill(seq.q, seq.k_pool, None, seq.prefix, seq.chunk, seq.bt, page_size=4,
                                    num_kv_heads=1, softmax_scale=0.2, kv_shared=True, head_dim_v=16)
    v_pool = np.ascontiguousarray(seq.k_pool[..., :16])
    o2, lse2 = oracle.chunked_prefill(seq.q, seq.k_pool, v_pool, seq.prefix, seq.chunk, seq.bt, page_size=4,
                                      num_kv_heads=1, softmax_scale=0.2)
    assert o.shape == (11, 6, 16)
    assert np.array_equal(o, o2) and np.array_equal(lse, lse2)


def test_rows_variant_matches_full():
    seq = Seq(4, 2, 8, 4, [10, 3, 0], [6, 9, 4], seed=51)
    o, lse = seq.run(0.5)
    samples = np.array([[0, 0], [5, 3], [6, 1], [14, 2], [15, 0], [18, 3]])
    qd = {int(t): seq.q[int(t)] for t in samples[:, 0]}
    for qarg in (seq.q, qd):
        o2, l2 = oracle.chunked_prefill_rows(qarg, seq.k_pool, seq.v_pool, seq.prefix, seq.chunk, seq.bt,
                                             samples, page_size=4, num_kv_heads=2, softmax_scale=0.5)
        assert np.max(np.abs(o2 - o[samples[:, 0], samples[:, 1]])) <= 1e-13
        assert np.max(np.abs(l2 - lse[samples[:, 0], samples[:, 1]])) <= 1e-13


def test_merge_of_disjoint_key_ranges_equals_full():
    rng = np.random.default_rng(9)
    n, m, d = 40, 12, 8
    K, V, Q = rng.standard_normal((n, d)), rng.standard_normal((n, d)), rng.standard_normal((m, d))
    limits = rng.integers(0, n, size=m)
    o_full, l_full = oracle.attention_rows(Q, K, V, limits, 0.4)
    cuts = [0, 7, 21, 22, n]
    o_parts, l_parts = [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        op = np.zeros((m, d))
        lp = np.full(m, -np.inf)
        for i in range(m):
            if limits[i] >= a:
                oo, ll = oracle.attention_rows(Q[i:i + 1], K[a:b], V[a:b], [limits[i] - a], 0.4)
                op[i], lp[i] = oo[0], ll[0]
        o_parts.append(op)
        l_parts.append(lp)
    o, l = oracle.merge_partials(o_parts, l_parts)
    assert np.max(np.abs(o - o_full)) <= 1e-12 and np.max(np.abs(l - l_full)) <= 1e-12


def test_needles_select_the_planted_value():
    # Every query head sees the same direction u; needles are keys along u whose strength grows
    # with position, so each query's output is the value of the last needle it can see.
    Hq, Hkv, d, B = 4, 1, 16, 4
    p, c = 12, 8
    seq = Seq(Hq, Hkv, d, B, [p], [c], seed=61)
    rng = np.random.default_rng(3)
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    seq.q[:] = f32_to_bf16_bits(np.tile(u * 4.0, (c, Hq, 1)))
    needles = sorted({0, B - 1, B, 2 * B - 1, 2 * B, p - 1, p, p + 3, p + c - 1})
    qv = oracle.bf16_bits_to_f64(seq.q[0, 0])
    for rank, j in enumerate(needles):
        want_logit = 20.0 * (rank + 1)
        kvec = u * (want_logit / (qv @ u))
        seq.k_pool[seq.bt[0, j // B], 0, j % B, :] = f32_to_bf16_bits(kvec)
    o, _ = seq.run(1.0)
    for i in range(c):
        last = max(j for j in needles if j <= p + i)
        v = oracle.bf16_bits_to_f64(seq.v_pool[seq.bt[0, last // B], 0, last % B])
        assert np.max(np.abs(o[i, :] - v[None, :])) <= 1e-6


# ------------------------------------------------------------------------------------------
# Append
# ------------------------------------------------------------------------------------------

def test_append_round_trip_and_untouched_slots():
    spec = wl.custom_wave(4, 2, 8, 8, 4, [5, 0, 8, 3], [6, 3, 0, 9], seed=2, bt_fill=10**9, bt_extra=2)
    t = wl.make_tensors(spec, seed=7)
    kp, vp = wl.to_bits(t["k_pool"]), wl.to_bits(t["v_pool"])
    kn, vn = wl.to_bits(t["k_new"]), wl.to_bits(t["v_new"])
    k1, v1 = oracle.append_kv(kp, vp, kn, vn, spec.prefix_lens, spec.chunk_lens, spec.block_table, 4)
    written = np.zeros(kp.shape[0] * 4, bool)
    cu = 0
    for r in range(spec.num_requests):
        p, c = int(spec.prefix_lens[r]), int(spec.chunk_lens[r])
        for i in range(c):
            page, slot = int(spec.block_table[r, (p + i) // 4]), (p + i) % 4
            assert np.array_equal(k1[page, :, slot], kn[cu + i]) and np.array_equal(v1[page, :, slot], vn[cu + i])
            written[page * 4 + slot] = True
        cu += c
    # brute-force scan of every slot: untouched ones keep their bits (including NaN poison)
    for page in range(kp.shape[0]):
        for slot in range(4):
            if not written[page * 4 + slot]:
                assert np.array_equal(k1[page, :, slot], kp[page, :, slot])
                assert np.array_equal(v1[page, :, slot], vp[page, :, slot])
    # inputs are not modified
    assert np.array_equal(kp, wl.to_bits(t["k_pool"]))


def test_entries_beyond_used_blocks_are_never_read():
    seq = Seq(4, 2, 8, 4, [5, 2], [3, 7], seed=71, bt_fill=-1)
    o, lse = seq.run(0.5)
    bt = seq.bt.copy()
    bt[bt < 0] = 2**30        # garbage past ceil(n/B) must be ignored
    o2, lse2 = oracle.chunked_prefill(seq.q, seq.k_pool, seq.v_pool, seq.prefix, seq.chunk, bt, page_size=4,
                                      num_kv_heads=2, softmax_scale=0.5)
    assert np.array_equal(o, o2)
    for r in range(2):
        assert oracle.num_blocks(int(seq.prefix[r] + seq.chunk[r]), 4) <= int((seq.bt[r] >= 0).sum())


def test_poisoned_pool_gives_finite_output():
    spec = wl.cfg1()
    t = wl.make_tensors(spec, seed=1000, poison=True)
    bits = {k: wl.to_bits(v) for k, v in t.items()}
    assert np.isnan(oracle.bf16_bits_to_f64(bits["k_pool"])).any()
    k1, v1 = oracle.append_kv(bits["k_pool"], bits["v_pool"], bits["k_new"], bits["v_new"], spec.prefix_lens,
                              spec.chunk_lens, spec.block_table, spec.page_size)
    o, lse = oracle.chunked_prefill(bits["q"], k1, v1, spec.prefix_lens, spec.chunk_lens, spec.block_table,
                                    page_size=spec.page_size, num_kv_heads=spec.num_kv_heads,
                                    softmax_scale=spec.softmax_scale)
    assert np.isfinite(o).all() and np.isfinite(lse).all()


# ------------------------------------------------------------------------------------------
# Teeth: planted mistakes in the oracle must fail the parity harness
# ------------------------------------------------------------------------------------------

def _run_spec(spec, bits, samples=None):
    k1, v1 = oracle.append_kv(bits["k_pool"], bits["v_pool"], bits["k_new"], bits["v_new"], spec.prefix_lens,
                              spec.chunk_lens, spec.block_table, spec.page_size)
    kw = dict(page_size=spec.page_size, num_kv_heads=spec.num_kv_heads, softmax_scale=spec.softmax_scale)
    if samples is None:
        o, l = oracle.chunked_prefill(bits["q"], k1, v1, spec.prefix_lens, spec.chunk_lens, spec.block_table, **kw)
        return o.reshape(-1, o.shape[-1]), l.reshape(-1)
    return oracle.chunked_prefill_rows(bits["q"], k1, v1, spec.prefix_lens, spec.chunk_lens, spec.block_table,
                                       samples, **kw)


def _mutants(monkeypatch, B):
    real_gather = oa.gather_positions
    real_rows = oa.attention_rows
    real_limit = oa._visible_limit

    def wrong_page(pool, bt_row, positions, page_size, kv_head):
        bt2 = np.array(bt_row, copy=True)
        last = int(np.max(positions)) // page_size
        if last >= 2:
            bt2[1] = bt_row[last]                      # logical block 1 read from the wrong page
        return real_gather(pool, bt2, positions, page_size, kv_head)

    def drop_page(q_rows, keys, values, limits, scale):
        keep = np.ones(keys.shape[0], bool)
        keep[B:2 * B] = False                              # logical block 1 ignored
        if keep.all() or not keep.any():
            return real_rows(q_rows, keys, values, limits, scale)
        idx = np.nonzero(keep)[0]
        lim = np.searchsorted(idx, np.asarray(limits), side="right") - 1
        return real_rows(q_rows, keys[idx], values[idx], np.maximum(lim, 0), scale)

    return {
        "wrong_page": ("gather_positions", wrong_page),
        "drop_page": ("attention_rows", drop_page),
        "diag_minus1": ("_visible_limit", lambda p, i: real_limit(p, i) - 1),
        "diag_plus1": ("_visible_limit", lambda p, i: real_limit(p, i) + 1),
    }


@pytest.mark.parametrize("which", ["wrong_page", "drop_page", "diag_minus1", "diag_plus1"])
def test_harness_rejects_mutant_oracle_cfg1(monkeypatch, which):
    spec = wl.cfg1()
    bits = {k: wl.to_bits(v) for k, v in wl.make_tensors(spec, seed=1000).items()}
    o_ref, l_ref = _run_spec(spec, bits)
    name, fn = _mutants(monkeypatch, spec.page_size)[which]
    monkeypatch.setattr(oa, name, fn)
    o_mut, l_mut = _run_spec(spec, bits)
    rep = _compare.report(o_mut, o_ref, l_mut, l_ref)
    assert not _compare.passes(rep), rep


@pytest.mark.parametrize("which", ["wrong_page", "drop_page", "diag_minus1"])
def test_harness_rejects_mutant_oracle_cfg2_sampled(monkeypatch, which):
    spec = wl.cfg2()
    bits = {k: wl.to_bits(v) for k, v in wl.make_tensors(spec, seed=2000).items()}
    rng = np.random.default_rng(0)
    cu = spec.cu_tokens
    toks = []
    for r in range(spec.num_requests):
        toks += [int(cu[r]), int(cu[r]) + 1, int(cu[r + 1]) - 1] + list(rng.integers(cu[r], cu[r + 1], 5))
    samples = np.array([[t, h] for t in toks for h in (0, 5, 31)])
    o_ref, l_ref = _run_spec(spec, bits, samples)
    name, fn = _mutants(monkeypatch, spec.page_size)[which]
    monkeypatch.setattr(oa, name, fn)
    o_mut, l_mut = _run_spec(spec, bits, samples)
    rep = _compare.report(o_mut, o_ref, l_mut, l_ref)
    assert not _compare.passes(rep), rep


@pytest.mark.parametrize("which", ["wrong_page", "drop_page", "diag_minus1", "diag_plus1"])
def test_harness_rejects_mutant_oracle_needles(monkeypatch, which):
    spec = wl.custom_wave(8, 2, 64, 64, 16, [48, 16], [40, 20], seed=5)
    t = wl.make_tensors(spec, seed=5)
    bits = {k: wl.to_bits(v) for k, v in t.items()}
    # needles: q rows of request 0 point along u; keys on every page's first/last slot and on the
    # chunk diagonal are scaled copies of u with growing strength
    rng = np.random.default_rng(1)
    u = rng.standard_normal(64)
    u /= np.linalg.norm(u)
    q = oracle.bf16_bits_to_f64(bits["q"])
    q[: 40] = u * 3.0
    bits["q"] = f32_to_bf16_bits(q)
    kn = oracle.bf16_bits_to_f64(bits["k_new"])
    kp = oracle.bf16_bits_to_f64(bits["k_pool"])
    pos = sorted({j for b in range(6) for j in (16 * b, 16 * b + 15) if j < 88} | {47, 48, 60, 87})
    for rank, j in enumerate(pos):
        vec = u * (6.0 * (rank + 1) / 3.0 / spec.softmax_scale)
        if j >= 48:
            kn[j - 48, :] = vec
        else:
            kp[spec.block_table[0, j // 16], :, j % 16] = vec
    bits["k_new"] = f32_to_bf16_bits(kn)
    bits["k_pool"] = f32_to_bf16_bits(kp)
    o_ref, l_ref = _run_spec(spec, bits)
    name, fn = _mutants(monkeypatch, spec.page_size)[which]
    monkeypatch.setattr(oa, name, fn)
    o_mut, l_mut = _run_spec(spec, bits)
    rep = _compare.report(o_mut, o_ref, l_mut, l_ref)
    assert not _compare.passes(rep), rep
    # even without the LSE check the needles make the output itself fail
    rep2 = _compare.report(o_mut, o_ref)
    assert not _compare.passes(rep2), rep2
