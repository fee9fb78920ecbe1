"""Pins of the fp64 KDA oracle against things other than itself (CPU only).

The recurrence (Eq. 2-3) is checked through properties the mathematics fixes, each reached by a
route that does not retype the update:

* retrieval: with beta_t = 1 and a unit key, reading the new state along k_t returns v_t exactly,
  whatever the decay and the previous state;
* interpolation: with a unit key and any beta_t, that read-out is (1 - beta_t) times the decayed
  old read-out plus beta_t v_t;
* pure decay: with beta = 0 the state is only scaled row-wise by the running product of the
  decays (numpy cumprod);
* plain causal linear attention: with no decay, beta = 1, a zero start and orthonormal keys the
  outputs equal tril(Q K^T) V (numpy matmul) and the final state is K^T V;
* gradient step: the erase-and-write is one gradient step of size beta_t on 1/2 ||S^T k - v||^2 at
  the decayed state (torch autograd, fp64);
* contraction: with zero values and unit keys the state's Frobenius norm never grows;
* resume: a request run as two chunks, the second resuming from the first's snapshot, equals the
  single chunk; idle lanes and untouched slots stay as they were.

Teeth: each planted mistake (decay after the erase, transposed read-out, erase sign, no decay,
beta dropped from the write or the erase, read-out before the update, decay on the value side,
resume from zero) makes at least one pin fail.
"""
import numpy as np
import pytest
import torch

from oracle import kda as ok
import workloads as wl


def unit_rows(rng, shape):
    x = rng.standard_normal(shape)
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def random_case(rng, c=12, H=3, dk=8, dv=8, unit_keys=True, beta=None, alpha=None):
    S0 = rng.standard_normal((H, dk, dv))
    q = rng.standard_normal((c, H, dk))
    k = unit_rows(rng, (c, H, dk)) if unit_keys else rng.standard_normal((c, H, dk))
    v = rng.standard_normal((c, H, dv))
    a = rng.uniform(0.0, 1.0, (c, H, dk)) if alpha is None else np.broadcast_to(alpha, (c, H, dk)).copy()
    b = rng.uniform(0.0, 1.0, (c, H)) if beta is None else np.broadcast_to(beta, (c, H)).copy()
    return S0, q, k, v, a, b


# --------------------------------------------------------------------------------------------
# Pins.  Each returns True when the (possibly mutated) oracle satisfies the property.
# --------------------------------------------------------------------------------------------

def pin_retrieval(seed=0):
    rng = np.random.default_rng(seed)
    S0, _, k, v, a, b = random_case(rng, beta=1.0)
    o, _ = ok.kda_recurrence(S0, k, k, v, a, b)          # query = key
    return np.abs(o - v).max() <= 1e-12


def pin_interpolation(seed=1):
    rng = np.random.default_rng(seed)
    S0, _, k, v, a, b = random_case(rng)
    o, _, states = ok.kda_recurrence(S0, k, k, v, a, b, keep_states=True)
    prev = np.concatenate([S0[None], states[:-1]])
    # (Diag(alpha_t) S_{t-1})^T k_t, through numpy matmul on each head
    old = np.stack([np.stack([(a[t, h][:, None] * prev[t, h]).T @ k[t, h] for h in range(k.shape[1])])
                    for t in range(k.shape[0])])
    want = (1.0 - b)[:, :, None] * old + b[:, :, None] * v
    return np.abs(o - want).max() <= 1e-12


def pin_pure_decay(seed=2):
    rng = np.random.default_rng(seed)
    S0, q, k, v, a, _ = random_case(rng, unit_keys=False, beta=0.0)
    o, S = ok.kda_recurrence(S0, q, k, v, a, np.zeros(q.shape[:2]))
    gamma = np.cumprod(a, axis=0)                                           # [c, H, d_k]
    want = np.einsum("hij,thi->thj", S0, gamma * q)
    return (np.abs(o - want).max() <= 1e-12 and
            np.abs(S - gamma[-1][:, :, None] * S0).max() <= 1e-12)


def pin_linear_attention(seed=3):
    rng = np.random.default_rng(seed)
    c, H, d = 10, 2, 16
    q = rng.standard_normal((c, H, d))
    v = rng.standard_normal((c, H, d))
    k = np.zeros((c, H, d))
    for h in range(H):
        Qm, _ = np.linalg.qr(rng.standard_normal((d, d)))
        k[:, h] = Qm[:c]                                   # orthonormal keys
    o, S = ok.kda_recurrence(np.zeros((H, d, d)), q, k, v, np.ones((c, H, d)), np.ones((c, H)))
    ok_all = True
    for h in range(H):
        want = np.tril(q[:, h] @ k[:, h].T) @ v[:, h]
        ok_all &= np.abs(o[:, h] - want).max() <= 1e-12
        ok_all &= np.abs(S[h] - k[:, h].T @ v[:, h]).max() <= 1e-12
    return bool(ok_all)


def pin_gradient_step(seed=4):
    rng = np.random.default_rng(seed)
    S0, q, k, v, a, b = random_case(rng, c=1, H=2, dk=6, dv=5)
    _, S1 = ok.kda_recurrence(S0, q, k, v, a, b)
    for h in range(2):
        Sd = torch.tensor(a[0, h][:, None] * S0[h], dtype=torch.float64, requires_grad=True)
        kk = torch.tensor(k[0, h], dtype=torch.float64)
        vv = torch.tensor(v[0, h], dtype=torch.float64)
        loss = 0.5 * ((Sd.T @ kk - vv) ** 2).sum()
        (grad,) = torch.autograd.grad(loss, Sd)
        want = (Sd - float(b[0, h]) * grad).detach().numpy()
        if np.abs(S1[h] - want).max() > 1e-12:
            return False
    return True


def pin_contraction(seed=5):
    rng = np.random.default_rng(seed)
    S0, q, k, _, a, b = random_case(rng, c=20)
    v = np.zeros((20, 3, 8))
    _, _, states = ok.kda_recurrence(S0, q, k, v, a, b, keep_states=True)
    norms = np.concatenate([[np.linalg.norm(S0, axis=(1, 2))], np.linalg.norm(states, axis=(2, 3))])
    return bool((np.diff(norms, axis=0) <= 1e-12).all())


def _wave_arrays(rng, c_total, H, dk, dv):
    q = wl.to_bits(torch.randn(c_total, H, dk, generator=torch.Generator().manual_seed(int(rng.integers(1 << 30))))
                   .to(torch.bfloat16))
    k = wl.to_bits(torch.randn(c_total, H, dk, generator=torch.Generator().manual_seed(int(rng.integers(1 << 30))))
                   .to(torch.bfloat16))
    v = wl.to_bits(torch.randn(c_total, H, dv, generator=torch.Generator().manual_seed(int(rng.integers(1 << 30))))
                   .to(torch.bfloat16))
    alpha = rng.uniform(0.5, 1.0, (c_total, H, dk)).astype(np.float32)
    beta = rng.uniform(0.0, 1.0, (c_total, H)).astype(np.float32)
    return q, k, v, alpha, beta


def pin_resume(seed=6):
    rng = np.random.default_rng(seed)
    H, dk, dv = 2, 8, 8
    c1, c2 = 7, 9
    q, k, v, alpha, beta = _wave_arrays(rng, c1 + c2, H, dk, dv)
    pool = rng.standard_normal((4, H, dk, dv)).astype(np.float32)
    # single chunk from slot 0 into slot 1
    o_one, p_one = ok.chunked_prefill(q, k, v, alpha, beta, pool, [c1 + c2], [0], [1])
    # two chunks: slot 0 -> slot 2, then slot 2 -> slot 2 (in place)
    o_a, p_a = ok.chunked_prefill(q[:c1], k[:c1], v[:c1], alpha[:c1], beta[:c1], pool, [c1], [0], [2])
    o_b, p_b = ok.chunked_prefill(q[c1:], k[c1:], v[c1:], alpha[c1:], beta[c1:], p_a.astype(np.float32), [c2],
                                  [2], [2])
    o_two = np.concatenate([o_a, o_b])
    # the fp32 round trip of the intermediate snapshot is the only rounding
    same_o = np.abs(o_two - o_one).max() <= 1e-4 * max(1.0, np.abs(o_one).max())
    same_s = np.abs(p_b[2] - p_one[1]).max() <= 1e-4 * max(1.0, np.abs(p_one[1]).max())
    untouched = np.array_equal(p_one[[0, 2, 3]], pool[[0, 2, 3]].astype(np.float64))
    return bool(same_o and same_s and untouched)


PINS = [pin_retrieval, pin_interpolation, pin_pure_decay, pin_linear_attention, pin_gradient_step,
        pin_contraction, pin_resume]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin):
    assert pin()


def test_resume_is_exact_in_fp64():
    """Resuming from an fp64 snapshot reproduces the single run to rounding (no fp32 hop)."""
    rng = np.random.default_rng(7)
    S0, q, k, v, a, b = random_case(rng, c=15, unit_keys=False)
    o, S = ok.kda_recurrence(S0, q, k, v, a, b)
    o1, S1 = ok.kda_recurrence(S0, q[:6], k[:6], v[:6], a[:6], b[:6])
    o2, S2 = ok.kda_recurrence(S1, q[6:], k[6:], v[6:], a[6:], b[6:])
    assert np.abs(np.concatenate([o1, o2]) - o).max() <= 1e-12
    assert np.abs(S2 - S).max() <= 1e-12


def test_cold_start_and_idle_lane():
    rng = np.random.default_rng(8)
    H, dk, dv = 2, 4, 4
    q, k, v, alpha, beta = _wave_arrays(rng, 5, H, dk, dv)
    pool = rng.standard_normal((3, H, dk, dv)).astype(np.float32)
    o, p = ok.chunked_prefill(q, k, v, alpha, beta, pool, [0, 5, 0], [0, -1, 1], [1, 2, 0])
    o_ref, S_ref = ok.kda_recurrence(np.zeros((H, dk, dv)), *[ok.bf16_bits_to_f64(x) for x in (q, k, v)],
                                     alpha.astype(np.float64), beta.astype(np.float64))
    assert np.abs(o - o_ref).max() == 0.0
    assert np.abs(p[2] - S_ref).max() == 0.0
    # idle lanes read and write nothing
    assert np.array_equal(p[[0, 1]], pool[[0, 1]].astype(np.float64))


def test_all_snapshots_read_before_any_write():
    """Request 0 writes the slot request 1 resumes from: request 1 must still see the old value."""
    rng = np.random.default_rng(9)
    H, dk, dv = 1, 4, 4
    q, k, v, alpha, beta = _wave_arrays(rng, 6, H, dk, dv)
    pool = rng.standard_normal((3, H, dk, dv)).astype(np.float32)
    o, _ = ok.chunked_prefill(q, k, v, alpha, beta, pool, [3, 3], [0, 1], [1, 2])
    o1, _ = ok.chunked_prefill(q[3:], k[3:], v[3:], alpha[3:], beta[3:], pool, [3], [1], [2])
    assert np.abs(o[3:] - o1).max() == 0.0


def test_head_subset_matches_full():
    rng = np.random.default_rng(10)
    H, dk, dv = 4, 4, 6
    q, k, v, alpha, beta = _wave_arrays(rng, 9, H, dk, dv)
    pool = rng.standard_normal((2, H, dk, dv)).astype(np.float32)
    o, p = ok.chunked_prefill(q, k, v, alpha, beta, pool, [4, 5], [0, -1], [1, 0])
    o2, p2 = ok.chunked_prefill(q, k, v, alpha, beta, pool, [4, 5], [0, -1], [1, 0], heads=[3, 1])
    assert np.array_equal(o[:, [3, 1]], o2)
    assert np.array_equal(p[:, [3, 1]], p2[:, [3, 1]])


def test_snapshot_size():
    """Eq. 4 for one layer: one d_k x d_v state per head, e.g. 4 MiB of fp32 for 64 heads of 128."""
    assert ok.snapshot_elements(64, 128, 128) * 4 == 4 * 1024 * 1024


# --------------------------------------------------------------------------------------------
# Teeth
# --------------------------------------------------------------------------------------------

def _m_decay_after(S, q, k, v, alpha, beta):
    along = np.einsum("hi,hij->hj", k, S)
    S1 = S - beta[:, None, None] * k[:, :, None] * along[:, None, :] + beta[:, None, None] * k[:, :, None] * v[:, None, :]
    S1 = alpha[:, :, None] * S1
    return S1, np.einsum("hij,hi->hj", S1, q)


def _mutant(**flags):
    def step(S, q, k, v, alpha, beta):
        dec = S if flags.get("no_decay") else (S * alpha[:, None, :] if flags.get("decay_cols")
                                               else alpha[:, :, None] * S)
        along = np.einsum("hi,hij->hj", k, dec)
        be = 1.0 if flags.get("no_beta_erase") else beta[:, None, None]
        bw = 1.0 if flags.get("no_beta_write") else beta[:, None, None]
        sign = 1.0 if flags.get("erase_sign") else -1.0
        S1 = dec + sign * be * k[:, :, None] * along[:, None, :] + bw * k[:, :, None] * v[:, None, :]
        src = S if flags.get("read_before") else S1
        o = (np.einsum("hij,hj->hi", src, q) if flags.get("read_transposed")
             else np.einsum("hij,hi->hj", src, q))
        return S1, o
    return step


MUTANTS = {
    "decay_after_erase": _m_decay_after,
    "transposed_readout": _mutant(read_transposed=True),
    "erase_sign": _mutant(erase_sign=True),
    "no_decay": _mutant(no_decay=True),
    "beta_dropped_from_write": _mutant(no_beta_write=True),
    "beta_dropped_from_erase": _mutant(no_beta_erase=True),
    "readout_before_update": _mutant(read_before=True),
    "decay_on_value_side": _mutant(decay_cols=True),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(name, monkeypatch):
    monkeypatch.setattr(ok, "kda_token", MUTANTS[name])

    def rejects(pin):
        try:
            return not pin()
        except ValueError:          # a shape error (value-side decay with d_k != d_v) also rejects
            return True

    failed = [p.__name__ for p in PINS if rejects(p)]
    assert failed, f"no pin rejects the mutant {name}"


def test_pins_reject_resume_from_zero(monkeypatch):
    real = ok.chunked_prefill

    def ignore_state_in(q, k, v, alpha, beta, pool, chunk_lens, state_in, state_out, heads=None):
        return real(q, k, v, alpha, beta, pool, chunk_lens, [-1] * len(state_in), state_out, heads)

    monkeypatch.setattr(ok, "chunked_prefill", ignore_state_in)
    assert not pin_resume()
