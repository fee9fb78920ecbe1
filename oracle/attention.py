"""fp64 reference for one wave of chunked prefill over a paged KV cache.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed, with the passages it follows:

* Paging (Preliminaries, "Reuse"): a request with n cached tokens and block size B occupies
  ceil(n / B) logical blocks whose physical pages need not be contiguous.  Logical position j
  lives in physical page ``block_table[r][j // B]`` at slot ``j % B``.
* Chunked prefill (Design of WavePP, "Waves and lanes"; A Minimum Implementation, steps 3-5):
  the uncached suffix of a request is cut into contiguous chunks.  Before a chunk executes, its
  freshly reserved suffix blocks are materialized; the chunk's K/V is written into them, and the
  chunk's queries then attend to the whole cached prefix plus the chunk itself, causally.
* Spans (Pipeline Scheduling, last paragraphs): each chunk is described by its request, its
  starting token (= the cached length p_r) and its length c_r; query i of the chunk sits at
  position p_r + i.
* Grouped-query and latent caches (Preliminaries, "Transformer Architectures"): several query
  heads share one KV head; a latent cache stores one shared vector per token from which both the
  keys and (here, its leading lanes) the values are read.

The attention itself is the textbook definition: for query position p_r + i and head h with KV
head g = h // G (G = Hq / Hkv), logits s_j = scale * <q, K(r, j)> for j in [0, p_r + i],
output = sum_j softmax(s)_j V(r, j), lse = log sum_j exp(s_j) (natural log).  The oracle
materializes the logits of a row tile, masks by selection, subtracts the exact row maximum and
normalizes; there is no online rescaling, blocking over keys or fusion.

Inputs are bf16 bit patterns (numpy uint16); they are widened exactly to fp64.
"""
from __future__ import annotations

import numpy as np


# ------------------------------------------------------------------------------------------
# Representation
# ------------------------------------------------------------------------------------------

def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact widening of bf16 bit patterns: a bf16 is the upper half of an IEEE fp32."""
    b = np.ascontiguousarray(bits).view(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def num_blocks(n: int, page_size: int) -> int:
    """ceil(n / B): logical blocks occupied by n tokens (Preliminaries, "Reuse")."""
    return -(-int(n) // int(page_size))


def gather_positions(pool, bt_row, positions, page_size, kv_head):
    """Pool rows for the given logical positions of one request through its block-table row.

    Only the blocks that the positions fall in are looked up; entries of the row beyond them
    are never read.
    """
    positions = np.asarray(positions, dtype=np.int64)
    pages = np.asarray(bt_row, dtype=np.int64)[positions // page_size]
    return pool[pages, kv_head, positions % page_size, :]


def _visible_limit(prefix_len: int, i):
    """Last key position a chunk query at index i may attend to: its own position p + i
    (causal, diagonal included)."""
    return prefix_len + np.asarray(i, dtype=np.int64)


# ------------------------------------------------------------------------------------------
# Append (materialization of the freshly reserved suffix blocks)
# ------------------------------------------------------------------------------------------

def append_kv(k_pool, v_pool, k_new, v_new, prefix_lens, chunk_lens, block_table, page_size):
    """Return copies of the pools with each chunk's K/V written at positions [p_r, p_r + c_r).

    A Minimum Implementation, step 4: the uncached suffix blocks are materialized before the chunk
    executes.  Token i of request r goes to page block_table[r][(p_r + i) // B], slot
    (p_r + i) % B, for every KV head.  Nothing else changes.  Works on bit patterns, so the result
    is bit-exact by construction.  ``v_pool``/``v_new`` are None for a shared latent cache.
    """
    k_out = np.array(k_pool, copy=True)
    v_out = None if v_pool is None else np.array(v_pool, copy=True)
    cu = 0
    for r in range(len(prefix_lens)):
        p, c = int(prefix_lens[r]), int(chunk_lens[r])
        if c:
            pos = p + np.arange(c, dtype=np.int64)
            pages = np.asarray(block_table[r], dtype=np.int64)[pos // page_size]
            slots = pos % page_size
            # pool[page, :, slot, :] = new[token, :, :] for every token of the chunk
            k_out[pages, :, slots, :] = k_new[cu:cu + c]
            if v_out is not None:
                v_out[pages, :, slots, :] = v_new[cu:cu + c]
        cu += c
    return k_out, v_out


# ------------------------------------------------------------------------------------------
# Attention
# ------------------------------------------------------------------------------------------

def attention_rows(q_rows, keys, values, limits, scale):
    """Softmax attention of query rows over keys 0..limit (inclusive) of one sequence.

    q_rows [m, d_qk], keys [n, d_qk], values [n, d_v] in fp64; limits [m] int.
    Returns o [m, d_v] and the natural-log LSE [m].
    """
    s = scale * (q_rows @ keys.T)                                  # [m, n]
    visible = np.arange(keys.shape[0])[None, :] <= np.asarray(limits)[:, None]
    s = np.where(visible, s, -np.inf)
    mx = s.max(axis=1)
    e = np.exp(s - mx[:, None])
    l = e.sum(axis=1)
    o = (e @ values) / l[:, None]
    return o, mx + np.log(l)


def _request_kv(k_pool, v_pool, bt_row, n, page_size, kv_head, kv_shared, head_dim_v):
    pos = np.arange(n, dtype=np.int64)
    k = bf16_bits_to_f64(gather_positions(k_pool, bt_row, pos, page_size, kv_head))
    if kv_shared:
        v = k[:, :head_dim_v]                     # values are the leading lanes of the latent
    else:
        v = bf16_bits_to_f64(gather_positions(v_pool, bt_row, pos, page_size, kv_head))
    return k, v


def chunked_prefill(q, k_pool, v_pool, prefix_lens, chunk_lens, block_table, *, page_size, num_kv_heads,
                    softmax_scale, kv_shared=False, head_dim_v=None, row_tile=256):
    """Attention of every chunk query of the wave; the pools must already hold the chunks' K/V.

    q [T, Hq, d_qk] bf16 bits, tokens packed by request in order; pools [P, Hkv, B, d] bf16 bits
    (``v_pool`` None when ``kv_shared``).  Returns o [T, Hq, d_v] fp64 and lse [T, Hq] fp64.
    """
    T, Hq, _ = q.shape
    G = Hq // num_kv_heads
    if head_dim_v is None:
        head_dim_v = (v_pool.shape[-1] if v_pool is not None else k_pool.shape[-1])
    o = np.zeros((T, Hq, head_dim_v), dtype=np.float64)
    lse = np.zeros((T, Hq), dtype=np.float64)
    cu = 0
    for r in range(len(prefix_lens)):
        p, c = int(prefix_lens[r]), int(chunk_lens[r])
        if c == 0:
            continue
        n = p + c
        for g in range(num_kv_heads):
            k, v = _request_kv(k_pool, v_pool, block_table[r], n, page_size, g, kv_shared, head_dim_v)
            for h in range(g * G, (g + 1) * G):
                for i0 in range(0, c, row_tile):
                    i1 = min(c, i0 + row_tile)
                    qr = bf16_bits_to_f64(q[cu + i0:cu + i1, h, :])
                    oo, ll = attention_rows(qr, k, v, _visible_limit(p, np.arange(i0, i1)), softmax_scale)
                    o[cu + i0:cu + i1, h, :] = oo
                    lse[cu + i0:cu + i1, h] = ll
        cu += c
    return o, lse


def chunked_prefill_rows(q, k_pool, v_pool, prefix_lens, chunk_lens, block_table, samples, *, page_size,
                         num_kv_heads, softmax_scale, kv_shared=False, head_dim_v=None):
    """The same result as :func:`chunked_prefill`, for selected (token, head) rows only.

    ``samples`` is an int array [m, 2] of (packed token index, query head).  ``q`` may be the full
    [T, Hq, d_qk] array or a dict {token: [Hq, d_qk] bits} holding at least the sampled tokens.
    Returns o [m, d_v] and lse [m].
    """
    samples = np.asarray(samples, dtype=np.int64).reshape(-1, 2)
    Hq = None
    cu = np.concatenate([[0], np.cumsum(np.asarray(chunk_lens, dtype=np.int64))])
    if head_dim_v is None:
        head_dim_v = (v_pool.shape[-1] if v_pool is not None else k_pool.shape[-1])
    o = np.zeros((len(samples), head_dim_v), dtype=np.float64)
    lse = np.zeros(len(samples), dtype=np.float64)
    req = np.searchsorted(cu, samples[:, 0], side="right") - 1
    groups = {}
    for idx, (t, h) in enumerate(samples):
        if Hq is None:
            Hq = (q[int(t)].shape[0] if isinstance(q, dict) else q.shape[1])
        g = int(h) // (Hq // num_kv_heads)
        groups.setdefault((int(req[idx]), g), []).append(idx)
    for (r, g), idxs in groups.items():
        p, c = int(prefix_lens[r]), int(chunk_lens[r])
        k, v = _request_kv(k_pool, v_pool, block_table[r], p + c, page_size, g, kv_shared, head_dim_v)
        idxs = np.asarray(idxs)
        toks, heads = samples[idxs, 0], samples[idxs, 1]
        qr = bf16_bits_to_f64(np.stack([q[int(t)][int(h)] for t, h in zip(toks, heads)]))
        oo, ll = attention_rows(qr, k, v, _visible_limit(p, toks - cu[r]), softmax_scale)
        o[idxs] = oo
        lse[idxs] = ll
    return o, lse


def probabilities(q, k_pool, prefix_lens, chunk_lens, block_table, request, head, *, page_size,
                  num_kv_heads, softmax_scale):
    """Attention weights [c_r, n_r] of one request and query head (for tiny inputs)."""
    Hq = q.shape[1]
    G = Hq // num_kv_heads
    cu = int(np.sum(np.asarray(chunk_lens[:request], dtype=np.int64)))
    p, c = int(prefix_lens[request]), int(chunk_lens[request])
    n = p + c
    k = bf16_bits_to_f64(gather_positions(k_pool, block_table[request], np.arange(n), page_size, head // G))
    qr = bf16_bits_to_f64(q[cu:cu + c, head, :])
    s = softmax_scale * (qr @ k.T)
    visible = np.arange(n)[None, :] <= _visible_limit(p, np.arange(c))[:, None]
    s = np.where(visible, s, -np.inf)
    e = np.exp(s - s.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def merge_partials(o_parts, lse_parts):
    """Combine attention results over disjoint key ranges into the result over their union.

    Each part s holds its normalized output o_s and log-sum-exp lse_s; a part that saw no key has
    lse_s = -inf.  The union has LSE = log sum_s exp(lse_s) and output sum_s exp(lse_s - LSE) o_s.
    """
    o_parts = np.asarray(o_parts, dtype=np.float64)
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    top = lse_parts.max(axis=0)
    w = np.exp(lse_parts - top[None, :])                    # exp(-inf) = 0 for empty parts
    tot = w.sum(axis=0)
    o_parts = np.where(np.isneginf(lse_parts)[..., None], 0.0, o_parts)
    o = np.einsum("sm,smd->md", w, o_parts) / tot[:, None]
    return o, top + np.log(tot)
