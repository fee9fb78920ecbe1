"""Seeded synthetic waves for chunked prefill of a KDA (gated delta-rule) layer.

Shared by the tests, the bench and the oracle harness.  It holds shapes, chunk lengths, snapshot
slot assignments and random values only; none of the recurrence's arithmetic lives here.

Request r of a wave runs c_r new tokens.  It resumes from the snapshot in slot state_in[r] (-1:
nothing cached, start from the zero state) and leaves its final state in slot state_out[r]
(Preliminaries: a recurrent layer resumes only from the exact state at its prefix boundary).

Value recipe (the paper gives no KDA widths or value distributions, so these are stand-ins):
* q and k: per token and head, a direction drawn uniformly on the unit sphere (an N(0, 1) vector
  divided by its norm), rounded to bf16;
* v: N(0, 1), rounded to bf16;
* beta: sigmoid of N(0, 1), fp32, in (0, 1);
* alpha: exp(-rate_h * softplus(z)), z ~ N(0, 1), fp32, with a per-head rate drawn log-uniformly
  from [rate_lo, rate_hi].  The default range [1/256, 1/2] gives decays from about 0.998 to
  about 0.5 per token.  The "extreme" recipe uses rates in [1, 16] and sets 1 % of the decays
  to exactly 0 (full reset of that channel);
* resumed snapshots: N(0, 1) * 0.25, fp32.  Slots that no request reads hold NaN in correctness
  runs (so that a stray read is loud) and 0 in timing runs.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


@dataclass
class KdaSpec:
    name: str
    num_heads: int
    head_dim_k: int
    head_dim_v: int
    num_slots: int
    chunk_lens: np.ndarray     # int32 [R]
    state_in: np.ndarray       # int32 [R], -1 = zero state
    state_out: np.ndarray      # int32 [R]
    rate_lo: float = 1.0 / 256
    rate_hi: float = 0.5
    extreme: bool = False
    notes: dict = field(default_factory=dict)

    @property
    def num_requests(self) -> int:
        return int(self.chunk_lens.shape[0])

    @property
    def total_tokens(self) -> int:
        return int(self.chunk_lens.sum())

    @property
    def cu_tokens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.chunk_lens, dtype=np.int64)]).astype(np.int64)

    def read_slots(self) -> np.ndarray:
        """Slots some active request resumes from."""
        m = (self.chunk_lens > 0) & (self.state_in >= 0)
        return np.unique(self.state_in[m])


def custom(num_heads, head_dim_k, head_dim_v, chunk_lens, state_in, state_out, num_slots=None, *,
           extreme=False, rate_lo=1.0 / 256, rate_hi=0.5, name="kda_custom") -> KdaSpec:
    chunk_lens = np.asarray(chunk_lens, dtype=np.int32)
    state_in = np.asarray(state_in, dtype=np.int32)
    state_out = np.asarray(state_out, dtype=np.int32)
    if num_slots is None:
        num_slots = int(max([0] + list(state_in + 1) + list(state_out + 1)))
    if extreme:
        rate_lo, rate_hi = 1.0, 16.0
    return KdaSpec(name=name, num_heads=num_heads, head_dim_k=head_dim_k, head_dim_v=head_dim_v,
                   num_slots=int(num_slots), chunk_lens=chunk_lens, state_in=state_in, state_out=state_out,
                   rate_lo=rate_lo, rate_hi=rate_hi, extreme=extreme)


def small(extreme=False) -> KdaSpec:
    """Six requests covering the cases: cold start, idle lane, resume in place, one token, exactly
    one 64-token block, and a ragged multi-block chunk resumed into another slot."""
    return custom(4, 128, 128, [40, 0, 130, 1, 64, 200], [-1, 3, 0, 1, -1, 2], [4, 5, 0, 6, 7, 8], 10,
                  extreme=extreme, name="kda_small" + ("_extreme" if extreme else ""))


def wave(num_heads=64) -> KdaSpec:
    """A 16,384-token wave of four 4,096-token chunks (two cold, two resumed in place), 64 heads
    of width 128."""
    return custom(num_heads, 128, 128, [4096] * 4, [-1, 0, -1, 1], [2, 0, 3, 1], 4, name="kda_wave")


def long(num_heads=64) -> KdaSpec:
    """One request with a 16,384-token chunk, resumed in place."""
    return custom(num_heads, 128, 128, [16384], [0], [0], 1, name="kda_long")


def short(num_heads=64) -> KdaSpec:
    """64 chunks of 256 tokens, every other one resumed; snapshot traffic is a large share."""
    R = 64
    state_in = np.where(np.arange(R) % 2 == 1, np.arange(R), -1)
    return custom(num_heads, 128, 128, [256] * R, state_in, np.arange(R) + R, 2 * R, name="kda_short")


def config(name: str) -> KdaSpec:
    table = {"kda_small": small, "kda_wave": wave, "kda_long": long, "kda_short": short,
             "kda_small_extreme": lambda: small(extreme=True)}
    return table[name]()


def make_tensors(spec: KdaSpec, seed: int, device="cpu", poison: bool = True) -> dict:
    """Draw q, k, v (bf16), alpha, beta (fp32) and the snapshot pool (fp32) for ``spec``.

    Shapes: q, k [T, H, d_k]; v [T, H, d_v]; alpha [T, H, d_k]; beta [T, H];
    state_pool [num_slots, H, d_k, d_v].
    """
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    T, H, dk, dv = spec.total_tokens, spec.num_heads, spec.head_dim_k, spec.head_dim_v

    def unit(shape):
        x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        return (x / x.norm(dim=-1, keepdim=True)).to(torch.bfloat16)

    q = unit((T, H, dk))
    k = unit((T, H, dk))
    v = torch.randn((T, H, dv), generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)
    beta = torch.sigmoid(torch.randn((T, H), generator=gen, device=device, dtype=torch.float32))
    u = torch.rand((H,), generator=gen, device=device, dtype=torch.float32)
    rate = torch.exp(math.log(spec.rate_lo) + u * (math.log(spec.rate_hi) - math.log(spec.rate_lo)))
    z = torch.randn((T, H, dk), generator=gen, device=device, dtype=torch.float32)
    alpha = torch.exp(-rate[None, :, None] * torch.nn.functional.softplus(z))
    if spec.extreme:
        reset = torch.rand((T, H, dk), generator=gen, device=device, dtype=torch.float32) < 0.01
        alpha = alpha.masked_fill(reset, 0.0)
    pool = torch.full((spec.num_slots, H, dk, dv), float("nan") if poison else 0.0, device=device,
                      dtype=torch.float32)
    for s in spec.read_slots():
        pool[int(s)] = 0.25 * torch.randn((H, dk, dv), generator=gen, device=device, dtype=torch.float32)
    return {"q": q, "k": k, "v": v, "alpha": alpha.contiguous(), "beta": beta.contiguous(), "state_pool": pool}
