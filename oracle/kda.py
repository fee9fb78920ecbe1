"""fp64 reference for chunked prefill of a Kimi Delta Attention (KDA) layer, with resume from a
recurrent-state snapshot and a snapshot at the chunk boundary.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed, with the passages it follows:

* Linear attention (Preliminaries, "Transformer Architectures", Eq. 1): the layer keeps a
  recurrent state S_t of fixed size that summarizes the prefix; each token updates it by a linear
  map plus an additive term, and its output is read from the updated state.
* KDA, single head (same subsection, Eq. 2 and Eq. 3): with a per-channel decay alpha_t (a vector
  of d_k entries in [0, 1]), a scalar write strength beta_t, key k_t (d_k), value v_t (d_v) and
  query q_t (d_k), the state S_t is a d_k x d_v matrix and

      S_t = (I - beta_t k_t k_t^T) Diag(alpha_t) S_{t-1} + beta_t k_t v_t^T,
      o_t = S_t^T q_t.

  The decay is applied first, then the component along k_t is erased with strength beta_t, then
  beta_t k_t v_t^T is written; the output reads the state after the token's own update.
* Resume (Preliminaries, "Reuse", the paragraphs on linear attention): a recurrent layer resumes
  after token r only from the state S_r itself; a later state cannot be rewound.  A chunk of c
  tokens of a request with r cached tokens therefore starts from the snapshot S_r (the zero state
  when nothing is cached) and leaves the snapshot S_{r+c} at the chunk boundary, from which the
  next chunk resumes.  A snapshot holds H * d_k * d_v elements per layer (Eq. 4).

Every head is independent.  The oracle runs the recurrence token by token in fp64 exactly as
written above: a decay of the state's rows, a rank-1 erase along k, a rank-1 write, and the
read-out.  There is no chunking, factorization or reordering.

Inputs are bf16 bit patterns (numpy uint16) for q, k, v and fp32 for alpha, beta and the state
pool; all are widened exactly to fp64.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_bits_to_f64


def kda_token(S, q, k, v, alpha, beta):
    """One token of Eq. 2-3 for a stack of independent heads.

    S [H, d_k, d_v]; q, k, alpha [H, d_k]; v [H, d_v]; beta [H].  Returns (S_t, o_t [H, d_v]).
    """
    decayed = alpha[:, :, None] * S                               # Diag(alpha_t) S_{t-1}
    along_k = np.einsum("hi,hij->hj", k, decayed)                   # k^T Diag(alpha) S_{t-1}
    S_new = decayed - beta[:, None, None] * k[:, :, None] * along_k[:, None, :]   # erase along k
    S_new = S_new + beta[:, None, None] * k[:, :, None] * v[:, None, :]          # write beta k v^T
    o = np.einsum("hij,hi->hj", S_new, q)                          # o_t = S_t^T q_t
    return S_new, o


def kda_recurrence(S0, q, k, v, alpha, beta, keep_states=False):
    """Run c tokens of one request from the state S0, token by token.

    S0 [H, d_k, d_v]; q, k, alpha [c, H, d_k]; v [c, H, d_v]; beta [c, H]; all fp64.
    Returns (o [c, H, d_v], S_c [H, d_k, d_v]) and, with ``keep_states``, every S_t as
    [c, H, d_k, d_v] as a third item.
    """
    S = np.array(S0, dtype=np.float64, copy=True)
    c = q.shape[0]
    o = np.zeros((c,) + v.shape[1:], dtype=np.float64)
    states = [] if keep_states else None
    for t in range(c):
        S, o[t] = kda_token(S, q[t], k[t], v[t], alpha[t], beta[t])
        if keep_states:
            states.append(S.copy())
    if keep_states:
        return o, S, (np.stack(states) if states else np.zeros((0,) + S.shape))
    return o, S


def chunked_prefill(q, k, v, alpha, beta, state_pool, chunk_lens, state_in, state_out, heads=None):
    """One wave of KDA chunked prefill.

    q, k [T, H, d_k] and v [T, H, d_v] bf16 bits, tokens packed by request in order; alpha
    [T, H, d_k] and beta [T, H] fp32; state_pool [slots, H, d_k, d_v] fp32.
    Request r runs its c_r tokens from the snapshot in slot state_in[r] (the zero state when
    state_in[r] < 0) and its final state becomes the snapshot in slot state_out[r].  Every
    snapshot is read before any is written.  A request with c_r = 0 is an idle lane: it reads and
    writes nothing.

    ``heads`` restricts the computation to a subset of heads (sampled parity at full size).
    Returns (o [T, len(heads), d_v] fp64, pool_after fp64 copy of the pool with the written
    slots holding the selected heads' final states).
    """
    T, H, _ = q.shape
    heads = np.arange(H) if heads is None else np.asarray(heads, dtype=np.int64)
    d_v = v.shape[2]
    o = np.zeros((T, len(heads), d_v), dtype=np.float64)
    pool_before = np.asarray(state_pool, dtype=np.float64)
    pool_after = pool_before.copy()
    cu = 0
    for r, c in enumerate(np.asarray(chunk_lens, dtype=np.int64)):
        c = int(c)
        if c == 0:
            continue
        sl = slice(cu, cu + c)
        if int(state_in[r]) >= 0:
            S0 = pool_before[int(state_in[r])][heads]
        else:
            S0 = np.zeros((len(heads),) + pool_before.shape[2:], dtype=np.float64)
        o[sl], S_end = kda_recurrence(
            S0,
            bf16_bits_to_f64(q[sl][:, heads]),
            bf16_bits_to_f64(k[sl][:, heads]),
            bf16_bits_to_f64(v[sl][:, heads]),
            np.asarray(alpha[sl][:, heads], dtype=np.float64),
            np.asarray(beta[sl][:, heads], dtype=np.float64),
        )
        pool_after[int(state_out[r]), heads] = S_end
        cu += c
    return o, pool_after


def snapshot_elements(num_heads, head_dim_k, head_dim_v):
    """Elements of one layer's snapshot: one d_k x d_v state per head (Eq. 4, one layer)."""
    return int(num_heads) * int(head_dim_k) * int(head_dim_v)
