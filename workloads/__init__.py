"""Seeded synthetic waves for chunked-prefill attention over a paged KV cache.

This module is shared by the tests, the bench and the oracle harness.  It holds
shapes, lengths, block tables and random values only: none of the attention or
append arithmetic lives here, so the oracle and the HIP path stay independent.

A *wave* (Design of WavePP, "Waves and lanes") is a ragged batch of request
chunks.  Request r has a cached prefix of p_r tokens and a new chunk of c_r
tokens; its n_r = p_r + c_r positions occupy ceil(n_r / B) logical blocks whose
physical pages are named by row r of the block table (Preliminaries, "Reuse").
The pages backing positions [p_r, n_r) are the freshly reserved suffix blocks
that the append fills before attention runs (A Minimum Implementation, steps
3-5).

Values are bf16 = round-to-nearest-even of fp32 N(0, 1) draws from a seeded
torch generator.  Pool slots that hold no cached token (free pages, page tails,
the not-yet-appended chunk slots) are filled with bf16 NaN in correctness runs
so that any read of them is loud, and with zeros in timing runs.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

BF16_NAN_BITS = 0x7FC0


@dataclass
class WaveSpec:
    """Static description of one wave: head shapes, page pool and per-request spans."""

    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim_qk: int
    head_dim_v: int
    page_size: int
    num_pages: int
    kv_shared: bool
    softmax_scale: float
    prefix_lens: np.ndarray          # int32 [R]
    chunk_lens: np.ndarray           # int32 [R]
    block_table: np.ndarray          # int32 [R, bt_stride]
    layers: int = 1
    notes: dict = field(default_factory=dict)

    @property
    def num_requests(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def total_tokens(self) -> int:
        return int(self.chunk_lens.sum())

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def cu_tokens(self) -> np.ndarray:
        """Offsets of each request's chunk in the packed token dimension, length R + 1."""
        return np.concatenate([[0], np.cumsum(self.chunk_lens, dtype=np.int64)]).astype(np.int64)

    @property
    def bt_stride(self) -> int:
        return int(self.block_table.shape[1])

    def pairs(self) -> np.ndarray:
        """Visible (query, key) pairs per request and head: c*p + c*(c+1)/2."""
        p = self.prefix_lens.astype(np.int64)
        c = self.chunk_lens.astype(np.int64)
        return c * p + c * (c + 1) // 2


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def budget_ladder(b0: int, b_min: int, block: int) -> list[int]:
    """Wave budgets from repeated halving, aligned down to the block size and floored
    at b_min (Pipeline Scheduling, Eq. 6).  Used only to draw chunk sizes."""
    out = [b0]
    while out[-1] > b_min:
        nxt = max(b_min, (out[-1] // 2) // block * block)
        out.append(nxt)
    return out


def _assign_pages(n_pages_per_req, num_pages, rng, shared_pages=0, bt_fill=-1, bt_extra=0):
    """Build a block table from one permutation of the pool.

    The first ``shared_pages`` logical blocks of every request map to the same
    physical pages; every other block gets a page of its own.
    """
    perm = rng.permutation(num_pages).astype(np.int32)
    cursor = 0
    shared = perm[cursor:cursor + shared_pages]
    cursor += shared_pages
    R = len(n_pages_per_req)
    stride = max(1, max(n_pages_per_req) + bt_extra) if R else 1
    bt = np.full((R, stride), bt_fill, dtype=np.int32)
    for r, n in enumerate(n_pages_per_req):
        k = min(shared_pages, n)
        bt[r, :k] = shared[:k]
        own = n - k
        if cursor + own > num_pages:
            raise ValueError("page pool too small for the requested wave")
        bt[r, k:n] = perm[cursor:cursor + own]
        cursor += own
    return bt


def custom_wave(num_q_heads, num_kv_heads, head_dim_qk, head_dim_v, page_size, prefix_lens, chunk_lens,
                *, kv_shared=False, softmax_scale=None, num_pages=None, seed=0, shared_prefix_pages=0,
                pool_slack=0.1, bt_fill=-1, bt_extra=0, name="custom") -> WaveSpec:
    """General wave builder used by the configs and by the tests."""
    prefix_lens = np.asarray(prefix_lens, dtype=np.int32)
    chunk_lens = np.asarray(chunk_lens, dtype=np.int32)
    B = page_size
    n_pages = [ceil_div(int(p) + int(c), B) for p, c in zip(prefix_lens, chunk_lens)]
    need = shared_prefix_pages + sum(max(0, n - shared_prefix_pages) for n in n_pages)
    if num_pages is None:
        num_pages = max(1, int(math.ceil(need * (1.0 + pool_slack))))
    rng = np.random.default_rng(seed)
    bt = _assign_pages(n_pages, num_pages, rng, shared_pages=shared_prefix_pages, bt_fill=bt_fill,
                       bt_extra=bt_extra)
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(head_dim_qk)
    return WaveSpec(name=name, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads, head_dim_qk=head_dim_qk,
                    head_dim_v=head_dim_v, page_size=B, num_pages=num_pages, kv_shared=kv_shared,
                    softmax_scale=float(softmax_scale), prefix_lens=prefix_lens, chunk_lens=chunk_lens,
                    block_table=bt)


# --------------------------------------------------------------------------------------------
# The paper-shaped configurations
# --------------------------------------------------------------------------------------------

def cfg1(seed: int = 1000) -> WaveSpec:
    """1 request: 8 query heads, 2 KV heads, d = 64, B = 16; 48 cached tokens on 3 shuffled
    pages of a 16-page pool, a 32-token chunk on 2 fresh pages; scale 1/sqrt(64)."""
    w = custom_wave(8, 2, 64, 64, 16, [48], [32], num_pages=16, seed=seed, name="cfg1")
    return w


def cfg2(seed: int = 2000) -> WaveSpec:
    """4 ragged requests: 32/8 heads, d = 128, B = 64; prefix uniform in [0, 4096] rounded down
    to whole pages, chunk 2048 each; 512-page pool, block tables from one permutation."""
    rng = np.random.default_rng(seed)
    prefix = (rng.integers(0, 4097, size=4) // 64) * 64
    w = custom_wave(32, 8, 128, 128, 64, prefix, [2048] * 4, num_pages=512, seed=seed + 1, name="cfg2")
    return w


def cfg3(seed: int = 3000) -> WaveSpec:
    """High prefix reuse: 32 requests share one 16384-token prefix (the same 256 physical pages
    in every block table), then a private suffix of 64*U{0..32} tokens; chunk sizes drawn from
    the halving ladder 4096 -> 512; 64/8 heads, d = 128, B = 64; pool = needed pages + 10 %."""
    rng = np.random.default_rng(seed)
    ladder = budget_ladder(4096, 512, 64)
    priv = 64 * rng.integers(0, 33, size=32)
    chunks = rng.choice(np.asarray(ladder), size=32)
    prefix = 16384 + priv
    w = custom_wave(64, 8, 128, 128, 64, prefix, chunks, shared_prefix_pages=256, seed=seed + 1, name="cfg3")
    w.notes["ladder"] = ladder
    return w


def cfg4(seed: int = 4000) -> WaveSpec:
    """Concurrency 128: lengths U{8192..32768}, prefix-hit fraction U[0, 0.9] rounded down to pages;
    a 16384-token wave budget is cut into ragged chunks (at least 128) across requests in admission
    order, each chunk starting at a random point of that request's suffix (mid-page starts).
    64/8 heads, d = 128, B = 64; the same wave runs through 4 layers with distinct tensors."""
    rng = np.random.default_rng(seed)
    L = rng.integers(8192, 32769, size=128)
    h = rng.uniform(0.0, 0.9, size=128)
    p_hit = (np.floor(h * L / 64) * 64).astype(np.int64)
    budget = 16384
    prefix, chunks = [], []
    for r in range(128):
        if budget < 128:
            break
        suffix = int(L[r] - p_hit[r])
        c = min(int(rng.integers(128, 4097)), budget, suffix)
        progress = int(rng.integers(0, suffix - c + 1))
        prefix.append(int(p_hit[r]) + progress)
        chunks.append(c)
        budget -= c
    w = custom_wave(64, 8, 128, 128, 64, prefix, chunks, seed=seed + 1, name="cfg4")
    w.layers = 4
    return w


def cfg5(seed: int = 5000) -> WaveSpec:
    """MLA-style latent attention (absorbed form): 128 query heads over one shared 576-wide latent
    (V = its first 512 lanes), B = 64; 8 requests with 131072 cached tokens and 8192-token chunks."""
    w = custom_wave(128, 1, 576, 512, 64, [131072] * 8, [8192] * 8, kv_shared=True, num_pages=17408,
                    seed=seed, name="cfg5")
    return w


def cfg6p(seed: int = 6000) -> WaveSpec:
    """The paper's short-suffix shape: 4 requests, 124992 cached tokens (page aligned) and a
    4096-token suffix each; 64/8 heads, d = 128, B = 64."""
    return custom_wave(64, 8, 128, 128, 64, [124992] * 4, [4096] * 4, seed=seed, name="cfg6p")


def small_chunk(chunk: int, seed: int = 7000) -> WaveSpec:
    """Gather-bound sweep: 8 requests with 16384..32768 cached tokens and tiny chunks."""
    rng = np.random.default_rng(seed + chunk)
    prefix = (rng.integers(16384, 32769, size=8) // 64) * 64
    return custom_wave(64, 8, 128, 128, 64, prefix, [chunk] * 8, seed=seed + chunk + 1,
                       name=f"small{chunk}")


CONFIGS = {"1": cfg1, "2": cfg2, "3": cfg3, "4": cfg4, "5": cfg5, "6p": cfg6p}


def config(name: str, seed: int | None = None) -> WaveSpec:
    name = str(name)
    if name.startswith("small"):
        return small_chunk(int(name[5:]))
    fn = CONFIGS[name]
    return fn() if seed is None else fn(seed)


# --------------------------------------------------------------------------------------------
# Tensors
# --------------------------------------------------------------------------------------------

def prefix_slot_counts(spec: WaveSpec) -> np.ndarray:
    """For every physical page, how many leading slots hold cached (prefix) tokens.

    Cached tokens of a request fill its logical blocks from slot 0; a page shared by several
    requests holds the longest of their cached runs on it.
    """
    B = spec.page_size
    cnt = np.zeros(spec.num_pages, dtype=np.int64)
    for r in range(spec.num_requests):
        p = int(spec.prefix_lens[r])
        nb = ceil_div(p, B)
        if nb == 0:
            continue
        pages = spec.block_table[r, :nb].astype(np.int64)
        fill = np.full(nb, B, dtype=np.int64)
        fill[-1] = p - (nb - 1) * B
        np.maximum.at(cnt, pages, fill)
    return cnt


def _randn_bf16(shape, gen, device, chunk_elems=1 << 28):
    import torch
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    n = flat.numel()
    pos = 0
    while pos < n:
        m = min(chunk_elems, n - pos)
        flat[pos:pos + m] = torch.randn(m, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)
        pos += m
    return out


def make_tensors(spec: WaveSpec, seed: int, device="cpu", poison: bool = True, layer: int = 0) -> dict:
    """Draw q, k_new, v_new and the page pools for one layer of ``spec``.

    Returns a dict of torch bf16 tensors: q [T, Hq, d_qk], k_new [T, Hkv, d_qk],
    v_new [T, Hkv, d_v] (None if kv_shared), k_pool [P, Hkv, B, d_qk],
    v_pool [P, Hkv, B, d_v] (None if kv_shared).  Slots of the pools that hold no cached token
    are NaN (poison=True) or 0.
    """
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed) + 100 * int(layer))
    T, Hq, Hkv = spec.total_tokens, spec.num_q_heads, spec.num_kv_heads
    dq, dv, B, P = spec.head_dim_qk, spec.head_dim_v, spec.page_size, spec.num_pages
    q = _randn_bf16((T, Hq, dq), gen, device)
    k_new = _randn_bf16((T, Hkv, dq), gen, device)
    v_new = None if spec.kv_shared else _randn_bf16((T, Hkv, dv), gen, device)
    k_pool = _randn_bf16((P, Hkv, B, dq), gen, device)
    v_pool = None if spec.kv_shared else _randn_bf16((P, Hkv, B, dv), gen, device)
    cnt = torch.as_tensor(prefix_slot_counts(spec), device=device)
    invalid = torch.arange(B, device=device)[None, :] >= cnt[:, None]          # [P, B]
    fill = torch.tensor(float("nan") if poison else 0.0, dtype=torch.bfloat16, device=device)
    for pool in (k_pool, v_pool):
        if pool is None:
            continue
        pool.masked_fill_(invalid[:, None, :, None], fill)
    return {"q": q, "k_new": k_new, "v_new": v_new, "k_pool": k_pool, "v_pool": v_pool}


def to_bits(t) -> np.ndarray:
    """bf16 torch tensor -> numpy uint16 array of its bit patterns (CPU copy)."""
    import torch
    if t is None:
        return None
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)
