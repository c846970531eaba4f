"""Pins of the float64 KDA oracle (Tab. 1 KDA row, Tab. 3) against what the
paper and the mathematics fix, each computed on a path independent of the
oracle's own loop: explicit factor matrices, the GDN row it reduces to, closed
forms, the composition law of Eq. (4) / Eq. (6).  CPU only.
"""

import numpy as np
import pytest

from oracle import gdn, kda


def _rel(x, ref):
    return np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-300)


def _tokens(seed, L, d_k, d_v, g_range=(-0.4, 0.0)):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((L, d_k))
    k = rng.standard_normal((L, d_k))
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    v = rng.standard_normal((L, d_v))
    beta = rng.uniform(0.0, 1.0, size=L)
    gate = rng.uniform(*g_range, size=(L, d_k))
    return q, k, v, beta, gate


def _factors(k, beta, gate):
    """Explicit per-token transitions of the KDA row of Tab. 1:
    T_t = (I - beta_t k_t k_t^T) diag(exp(g_t))."""
    d = k.shape[1]
    return [(np.eye(d) - beta[t] * np.outer(k[t], k[t])) @ np.diag(np.exp(gate[t]))
            for t in range(len(beta))]


@pytest.mark.parametrize("with_s0", [False, True])
def test_kda_recurrence_matches_explicit_factor_sums(with_s0):
    """Brute force of Eq. (2): S_t = (prod_{r<=t} T_r) S_0 + sum_s (prod_{s<r<=t} T_r) u_s,
    o_t = S_t^T q_t, with explicit d x d factor matrices (d = 5, L = 9)."""
    q, k, v, beta, gate = _tokens(1, 9, 5, 3)
    rng = np.random.default_rng(2)
    S0 = rng.standard_normal((5, 3)) if with_s0 else None
    o, S = kda.kda_recurrence(q, k, v, beta, gate, S0=S0)
    T = _factors(k, beta, gate)
    for t in range(9):
        St = np.zeros((5, 3)) if S0 is None else S0.copy()
        P = np.eye(5)
        for r in range(t + 1):
            P = T[r] @ P
        St = P @ St
        for s in range(t + 1):
            Ps = np.eye(5)
            for r in range(s + 1, t + 1):
                Ps = T[r] @ Ps
            St = St + Ps @ (beta[s] * np.outer(k[s], v[s]))
        assert _rel(o[t], St.T @ q[t]) < 1e-12
    assert _rel(S, St) < 1e-12


def test_kda_operator_equals_ordered_factor_product():
    """Tab. 3: T_C = prod_t (I - beta_t k_t k_t^T) diag(g_t), later tokens on the left."""
    _, k, _, beta, gate = _tokens(3, 11, 6, 2)
    P = np.eye(6)
    for M in _factors(k, beta, gate):
        P = M @ P
    assert _rel(kda.kda_transition_product(k, beta, gate), P) < 1e-12
    # the reversed order is a different matrix (the pin can fail)
    R = np.eye(6)
    for M in _factors(k, beta, gate)[::-1]:
        R = M @ R
    assert _rel(R, P) > 1e-3


def test_kda_with_channel_uniform_gates_is_gdn():
    """With the same gate on every channel, diag(exp(g_t)) = alpha_t I commutes
    with the erasure, so the KDA row is the GDN row of Tab. 1 (whose oracle is
    pinned on its own)."""
    q, k, v, beta, gate = _tokens(4, 40, 8, 5)
    a = gate[:, 0]
    g = np.repeat(a[:, None], 8, axis=1)
    o1, S1 = kda.kda_recurrence(q, k, v, beta, g)
    o2, S2 = gdn.recurrence(q, k, v, beta, a)
    assert _rel(o1, o2) < 1e-12 and _rel(S1, S2) < 1e-12
    P_hat, ld = gdn.segment_operator(k, beta, a)
    assert _rel(kda.kda_transition_product(k, beta, g), np.exp(ld) * P_hat) < 1e-12


def test_kda_beta_zero_is_the_diagonal_family_without_writes():
    """beta = 0 removes both the erasure and the write: S stays 0 from a zero
    start, S_0 decays channel by channel, and T_C = diag(exp(sum_t g_t))."""
    q, k, v, _, gate = _tokens(5, 17, 6, 4)
    beta = np.zeros(17)
    o, S = kda.kda_recurrence(q, k, v, beta, gate)
    assert np.all(o == 0) and np.all(S == 0)
    S0 = np.random.default_rng(6).standard_normal((6, 4))
    _, S = kda.kda_recurrence(q, k, v, beta, gate, S0=S0)
    assert _rel(S, np.exp(gate.sum(axis=0))[:, None] * S0) < 1e-13
    assert _rel(kda.kda_transition_product(k, beta, gate), np.diag(np.exp(gate.sum(axis=0)))) < 1e-13


def test_kda_orthonormal_keys_closed_form():
    """Keys e_{c_t} (distinct basis vectors) and beta_t = 1: each token erases
    row c_t of the gated state and writes v_t there, so row c of S_L is the last
    v_t written to it, times the gates of channel c applied after that token."""
    L, d, dv = 6, 8, 3
    rng = np.random.default_rng(7)
    rows = [2, 5, 0, 7, 3, 6]
    k = np.eye(d)[rows]
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, dv))
    gate = rng.uniform(-0.5, 0.0, size=(L, d))
    S0 = rng.standard_normal((d, dv))
    _, S = kda.kda_recurrence(q, k, v, np.ones(L), gate, S0=S0)
    ref = np.exp(gate.sum(axis=0))[:, None] * S0
    for t, c in enumerate(rows):
        ref[c] = v[t] * np.exp(gate[t + 1:, c].sum())
    assert _rel(S, ref) < 1e-13


def test_kda_tuples_compose_to_the_concatenation():
    """Eq. (4) / Eq. (6): the tuples of segments A and B, composed behind a
    prefix state with the GDN composition (T_i = exp(log_decay_i) P_hat_i),
    give the recurrence over prefix + A + B; the seam from the composed state
    gives the first outputs of B."""
    q, k, v, beta, gate = _tokens(8, 150, 6, 4)
    S0 = np.random.default_rng(9).standard_normal((6, 4))
    cu = [0, 70, 150]
    b = kda.kda_build_segments(q[:, None], k[:, None], v[:, None], beta[:, None], gate[:, None],
                               cu)
    S_out, S_inc = gdn.compose(b["P_hat"], b["log_decay"], b["S_seg"], [0, 1], [0, 2],
                               S_prefix=S0[None, None])
    o_full, S_full = kda.kda_recurrence(q, k, v, beta, gate, S0=S0)
    assert _rel(S_out[0, 0], S_full) < 1e-12
    o_seam, S_post = kda.kda_seam(q[:, None], k[:, None], v[:, None], beta[:, None],
                                  gate[:, None], [70], [80], 16, S_inc[1:2])
    assert _rel(o_seam[0, :, 0], o_full[70:86]) < 1e-12
    _, S_86 = kda.kda_recurrence(q[:86], k[:86], v[:86], beta[:86], gate[:86], S0=S0)
    assert _rel(S_post[0, 0], S_86) < 1e-12
    # naive addition of the segment states is wrong (the pin can fail)
    assert _rel(b["S_seg"][0, 0] + b["S_seg"][1, 0], S_full) > 1e-2


def test_kda_operator_split_is_the_per_token_gate_maximum():
    """The oracle's scalar split of T_C (Tab. 3 fixes only T_C): each token's
    factor is divided by exp(max_c g_tc).  Hand-computed log_decay on a case
    with known per-token maxima; exp(log_decay) P_hat equals the explicit
    factor product; and P_hat stays in range where T_C itself underflows
    float64 (the split can fail: without it the product is 0)."""
    L, d = 70, 3
    gate = np.zeros((L, d))
    gate[:, 0] = -0.2
    gate[:, 1] = -0.05          # the largest channel of every token
    gate[:, 2] = -1.0
    k = np.eye(d)[np.arange(L) % d]
    beta = np.full(L, 0.5)
    b = kda.kda_build_segments(np.zeros((L, 1, d)), k[:, None], np.zeros((L, 1, 2)),
                               beta[:, None], gate[:, None], [0, L])
    assert abs(b["log_decay"][0, 0] - L * -0.05) < 1e-13
    T_C = kda.kda_transition_product(k, beta, gate)
    assert _rel(np.exp(b["log_decay"][0, 0]) * b["P_hat"][0, 0], T_C) < 1e-13
    F = np.eye(d)
    for t in range(L):
        F = (np.eye(d) - beta[t] * np.outer(k[t], k[t])) @ np.diag(np.exp(gate[t])) @ F
    assert _rel(T_C, F) < 1e-13
    # 4000 tokens of channel-uniform gates near -0.3 and one fixed unit key:
    # T_C ~ exp(-1200) underflows float64 (to zeros and denormals), while
    # P_hat = I - (1 - (1 - beta)^L) k k^T in closed form
    rng = np.random.default_rng(3)
    Lh = 4000
    gh = np.repeat(-0.3 + 0.01 * rng.standard_normal((Lh, 1)), d, axis=1)
    kv = rng.standard_normal(d)
    kv /= np.linalg.norm(kv)
    kh = np.tile(kv, (Lh, 1))
    ld, P = kda.kda_operator(kh, np.full(Lh, 0.5), gh)
    assert np.max(np.abs(kda.kda_transition_product(kh, np.full(Lh, 0.5), gh))) < 1e-300
    assert abs(ld - np.sum(gh[:, 0])) < 1e-9
    assert _rel(P, np.eye(d) - (1.0 - 0.5 ** Lh) * np.outer(kv, kv)) < 1e-12
