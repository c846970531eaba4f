"""Pins of the float64 oracle against what the paper and the mathematics fix.

Each check is computed independently of the oracle's own code path (explicit
factor matrices, closed forms, printed table values, brute force), so that a
dropped term, a wrong sign or index, a transposed operand or a reversed product
order in the oracle fails at least one of them.  CPU only.
"""

import os

import numpy as np
import pytest

import oracle
from oracle import gdn


def _rng(seed):
    return np.random.default_rng(seed)


def _tokens(rng, L, d_k, d_v, unit=True, beta_range=(0.0, 1.0), a_range=(-0.3, 0.0)):
    q = rng.standard_normal((L, d_k))
    k = rng.standard_normal((L, d_k))
    if unit:
        k /= np.linalg.norm(k, axis=1, keepdims=True)
        q /= np.linalg.norm(q, axis=1, keepdims=True)
    v = rng.standard_normal((L, d_v))
    beta = rng.uniform(*beta_range, size=L)
    a = rng.uniform(*a_range, size=L)
    return q, k, v, beta, a


def _factors(k, beta, a):
    """Explicit per-token transitions T_t = alpha_t (I - beta_t k_t k_t^T)
    (Tab. 1, GDN row)."""
    d = k.shape[1]
    return [np.exp(a[t]) * (np.eye(d) - beta[t] * np.outer(k[t], k[t]))
            for t in range(len(beta))]


def _left_product(mats, d):
    """prod with later factors on the left: M_n ... M_1 (Eq. 4 / Eq. 6 notation)."""
    P = np.eye(d)
    for M in mats:
        P = M @ P
    return P


def _rel(x, ref):
    return np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-300)


# --------------------------------------------------------------------------
# Brute force of Eq. (2): S_t = sum_s (prod_{r=s+1..t} T_r) u_s (+ carried S_0)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("with_s0", [False, True])
def test_recurrence_matches_explicit_factor_sums(with_s0):
    rng = _rng(1)
    L, d_k, d_v = 24, 8, 6           # d_k != d_v catches a transposed read-out
    q, k, v, beta, a = _tokens(rng, L, d_k, d_v, unit=False, beta_range=(0.0, 1.5))
    S0 = rng.standard_normal((d_k, d_v)) if with_s0 else None
    T = _factors(k, beta, a)
    u = [beta[t] * np.outer(k[t], v[t]) for t in range(L)]
    o_ref = np.zeros((L, d_v))
    for t in range(L):
        S_t = np.zeros((d_k, d_v)) if S0 is None else _left_product(T[:t + 1], d_k) @ S0
        for s in range(t + 1):
            S_t = S_t + _left_product(T[s + 1:t + 1], d_k) @ u[s]
        o_ref[t] = q[t] @ S_t          # o_t^T = q_t^T S_t, the state after the write
    o, S = oracle.recurrence(q, k, v, beta, a, S0=S0)
    assert _rel(o, o_ref) < 1e-12
    assert _rel(S, S_t) < 1e-12


def test_operator_equals_ordered_factor_product():
    """Sec. 5 construction identity: (prod_t T_t) I = T_C, later tokens on the
    left; Tab. 3 GDN closed form (prod g_t) prod (I - beta k k^T)."""
    rng = _rng(2)
    L, d = 20, 7
    _, k, _, beta, a = _tokens(rng, L, d, d)
    T = _factors(k, beta, a)
    T_C = _left_product(T, d)
    P_hat, log_decay = oracle.segment_operator(k, beta, a)
    assert abs(log_decay - a.sum()) < 1e-12
    assert _rel(np.exp(log_decay) * P_hat, T_C) < 1e-12
    # the reversed order is a different matrix: the check above can tell them apart
    T_rev = _left_product(T[::-1], d)
    assert _rel(T_rev, T_C) > 1e-3
    # decay-free factor on its own
    P_ref = _left_product([np.eye(d) - beta[t] * np.outer(k[t], k[t]) for t in range(L)], d)
    assert _rel(P_hat, P_ref) < 1e-12


# --------------------------------------------------------------------------
# Special cases named by the problem statement
# --------------------------------------------------------------------------

def test_beta_zero_gives_pure_decay():
    rng = _rng(3)
    L, d = 30, 9
    q, k, v, _, a = _tokens(rng, L, d, d)
    beta = np.zeros(L)
    P_hat, ld = oracle.segment_operator(k, beta, a)
    assert np.array_equal(P_hat, np.eye(d))
    assert abs(ld - a.sum()) < 1e-12
    o, S = oracle.recurrence(q, k, v, beta, a)
    assert np.all(S == 0) and np.all(o == 0)


def test_alpha_one_beta_zero_is_identity():
    rng = _rng(4)
    L, d = 17, 5
    q, k, v, _, _ = _tokens(rng, L, d, d)
    P_hat, ld = oracle.segment_operator(k, np.zeros(L), np.zeros(L))
    assert ld == 0.0
    assert np.array_equal(np.exp(ld) * P_hat, np.eye(d))
    S0 = rng.standard_normal((d, d))
    _, S = oracle.recurrence(q, k, v, np.zeros(L), np.zeros(L), S0=S0)
    assert np.array_equal(S, S0)


def test_unit_key_beta_one_factor_is_idempotent():
    rng = _rng(5)
    d = 11
    kk = rng.standard_normal(d)
    kk /= np.linalg.norm(kk)
    P1, _ = oracle.segment_operator(kk[None, :], np.ones(1), np.zeros(1))
    assert _rel(P1 @ P1, P1) < 1e-12
    # a segment repeating that token (alpha = 1) has the same operator as one token
    P5, _ = oracle.segment_operator(np.tile(kk, (5, 1)), np.ones(5), np.zeros(5))
    assert _rel(P5, P1) < 1e-12
    # and it is the orthogonal projector onto k's complement
    assert _rel(P1, np.eye(d) - np.outer(kk, kk)) < 1e-12


# --------------------------------------------------------------------------
# Closed forms
# --------------------------------------------------------------------------

def test_same_unit_key_closed_form():
    rng = _rng(6)
    L, d_k, d_v = 40, 10, 7
    q, _, v, beta, a = _tokens(rng, L, d_k, d_v)
    kk = rng.standard_normal(d_k)
    kk /= np.linalg.norm(kk)
    k = np.tile(kk, (L, 1))
    P_hat, _ = oracle.segment_operator(k, beta, a)
    P_ref = np.eye(d_k) - (1.0 - np.prod(1.0 - beta)) * np.outer(kk, kk)
    assert _rel(P_hat, P_ref) < 1e-12
    # S_t = k s_t^T with s_t = alpha_t (1 - beta_t) s_{t-1} + beta_t v_t; o_t = (q_t.k) s_t
    s = np.zeros(d_v)
    o_ref = np.zeros((L, d_v))
    for t in range(L):
        s = np.exp(a[t]) * (1.0 - beta[t]) * s + beta[t] * v[t]
        o_ref[t] = (q[t] @ kk) * s
    o, S = oracle.recurrence(q, k, v, beta, a)
    assert _rel(S, np.outer(kk, s)) < 1e-12
    assert _rel(o, o_ref) < 1e-12


def test_orthonormal_keys_closed_form():
    rng = _rng(7)
    d_k, d_v = 12, 5
    L = d_k
    Qm, _ = np.linalg.qr(rng.standard_normal((d_k, d_k)))
    k = Qm.T                                    # rows orthonormal
    q, _, v, beta, a = _tokens(rng, L, d_k, d_v)
    P_hat, _ = oracle.segment_operator(k, beta, a)
    P_ref = np.eye(d_k) - sum(beta[t] * np.outer(k[t], k[t]) for t in range(L))
    assert _rel(P_hat, P_ref) < 1e-12
    S_ref = sum(np.exp(a[t + 1:].sum()) * beta[t] * np.outer(k[t], v[t]) for t in range(L))
    _, S = oracle.recurrence(q, k, v, beta, a)
    assert _rel(S, S_ref) < 1e-12


# --------------------------------------------------------------------------
# Composition: Eq. (4), Eq. (6), associativity, naive addition (Eq. 3 / Eq. 5)
# --------------------------------------------------------------------------

def _concat_run(parts):
    q = np.concatenate([p[0] for p in parts])
    k = np.concatenate([p[1] for p in parts])
    v = np.concatenate([p[2] for p in parts])
    b = np.concatenate([p[3] for p in parts])
    a = np.concatenate([p[4] for p in parts])
    return q, k, v, b, a


def test_true_splice_two_segments():
    """Eq. (4): S_{C1C2|0} = T_{C2} S_{C1|0} + S_{C2|0}."""
    rng = _rng(8)
    d_k, d_v = 9, 6
    A = _tokens(rng, 33, d_k, d_v)
    B = _tokens(rng, 21, d_k, d_v)
    _, S_A = oracle.recurrence(*A)
    _, S_B = oracle.recurrence(*B)
    P_B, g_B = oracle.segment_operator(B[1], B[3], B[4])
    _, S_AB = oracle.recurrence(*_concat_run([A, B]))
    assert _rel(np.exp(g_B) * P_B @ S_A + S_B, S_AB) < 1e-12


def _ragged_case(rng, lens, d_k, d_v, h_qk=1, h_v=1, a_range=(-0.05, 0.0)):
    T = int(sum(lens))
    q = rng.standard_normal((T, h_qk, d_k))
    k = rng.standard_normal((T, h_qk, d_k))
    q /= np.linalg.norm(q, axis=2, keepdims=True)
    k /= np.linalg.norm(k, axis=2, keepdims=True)
    v = rng.standard_normal((T, h_v, d_v))
    beta = rng.uniform(0, 1, size=(T, h_v))
    a = rng.uniform(*a_range, size=(T, h_v))
    cu = np.concatenate([[0], np.cumsum(lens)])
    return q, k, v, beta, a, cu


def test_compose_behind_prefix_equals_concatenation_and_seams():
    """n segments behind a prefix composed by Eq. (6) equal the sequential
    recurrence over the concatenation; the state entering each segment equals the
    recurrence state at that boundary; the seam rescan from it reproduces the
    concatenation's outputs and states over each segment's first w tokens."""
    rng = _rng(9)
    lens = [37, 5, 64, 19]
    pre_len = 29
    d_k, d_v, h = 8, 10, 2
    q, k, v, beta, a, cu = _ragged_case(rng, [pre_len] + lens, d_k, d_v, h_qk=1, h_v=h,
                                        a_range=(-0.02, 0.0))
    seg_cu = cu[1:] - pre_len
    segs = slice(pre_len, None)
    built = oracle.build_segments(q[segs], k[segs], v[segs], beta[segs], a[segs], seg_cu)
    S_prefix = np.zeros((1, h, d_k, d_v))
    for hh in range(h):
        _, S_prefix[0, hh] = oracle.recurrence(q[:pre_len, 0], k[:pre_len, 0],
                                               v[:pre_len, hh], beta[:pre_len, hh],
                                               a[:pre_len, hh])
    order = np.arange(len(lens))
    S_out, S_inc = oracle.compose(built["P_hat"], built["log_decay"], built["S_seg"],
                                  order, [0, len(lens)], S_prefix=S_prefix)
    w = 8
    o_seam, S_post = oracle.seam(q[segs], k[segs], v[segs], beta[segs], a[segs],
                                 seg_cu[:-1], np.diff(seg_cu), w, S_inc)
    for hh in range(h):
        o_full, S_full = oracle.recurrence(q[:, 0], k[:, 0], v[:, hh], beta[:, hh], a[:, hh])
        assert _rel(S_out[0, hh], S_full) < 1e-11
        for j, L in enumerate(lens):
            start = pre_len + int(seg_cu[j])
            _, S_b = oracle.recurrence(q[:start, 0], k[:start, 0], v[:start, hh],
                                       beta[:start, hh], a[:start, hh])
            assert _rel(S_inc[j, hh], S_b) < 1e-11
            we = min(w, L)
            assert _rel(o_seam[j, :we, hh], o_full[start:start + we]) < 1e-11
            assert np.all(np.isnan(o_seam[j, we:, hh]))
            _, S_w = oracle.recurrence(q[:start + we, 0], k[:start + we, 0],
                                       v[:start + we, hh], beta[:start + we, hh],
                                       a[:start + we, hh])
            assert _rel(S_post[j, hh], S_w) < 1e-11


def test_compose_equals_literal_eq6_sum():
    """The closed sum of Eq. (6) written out term by term."""
    rng = _rng(10)
    n, d_k, d_v = 5, 6, 4
    T = [np.exp(rng.uniform(-0.5, 0)) * (np.eye(d_k) + 0.3 * rng.standard_normal((d_k, d_k)))
         for _ in range(n)]
    S = [rng.standard_normal((d_k, d_v)) for _ in range(n)]
    S_S = rng.standard_normal((d_k, d_v))
    ref = _left_product(T, d_k) @ S_S
    for i in range(n):
        ref = ref + _left_product(T[i + 1:], d_k) @ S[i]
    P_hat = np.stack([T[i] for i in range(n)])[:, None]
    ld = np.zeros((n, 1))
    S_seg = np.stack(S)[:, None]
    S_out, _ = oracle.compose(P_hat, ld, S_seg, np.arange(n), [0, n], S_prefix=S_S[None, None])
    assert _rel(S_out[0, 0], ref) < 1e-12
    # a permuted order gives a different state (order matters)
    S_perm, _ = oracle.compose(P_hat, ld, S_seg, np.arange(n)[::-1], [0, n],
                               S_prefix=S_S[None, None])
    assert _rel(S_perm[0, 0], ref) > 1e-3


def test_compose_associativity():
    """(P_c P_b) P_a: merging two tuples first, (P_b, S_b) o (P_a, S_a) =
    (P_b P_a, P_b S_a + S_b), gives the same composed state."""
    rng = _rng(11)
    d = 7
    tup = []
    for _ in range(3):
        _, k, v, beta, a = _tokens(rng, 15, d, d)
        P, g = oracle.segment_operator(k, beta, a)
        _, S = oracle.recurrence(np.zeros((15, d)), k, v, beta, a)
        tup.append((np.exp(g) * P, S))
    S0 = rng.standard_normal((d, d))
    (Pa, Sa), (Pb, Sb), (Pc, Sc) = tup
    Pcb, Scb = Pc @ Pb, Pc @ Sb + Sc
    P_hat = np.stack([Pa, Pb, Pc])[:, None]
    out, _ = oracle.compose(P_hat, np.zeros((3, 1)), np.stack([Sa, Sb, Sc])[:, None],
                            [0, 1, 2], [0, 3], S_prefix=S0[None, None])
    assert _rel(out[0, 0], Pcb @ (Pa @ S0 + Sa) + Scb) < 1e-12


def test_naive_addition_fails_for_gdn():
    """Eq. (3) summing end-states is not the GDN end-state (Eq. 5 error)."""
    rng = _rng(12)
    d = 16
    A = _tokens(rng, 64, d, d, a_range=(-2.0 ** -10, -2.0 ** -10))
    B = _tokens(rng, 64, d, d, a_range=(-2.0 ** -10, -2.0 ** -10))
    _, S_A = oracle.recurrence(*A)
    _, S_B = oracle.recurrence(*B)
    _, S_AB = oracle.recurrence(*_concat_run([A, B]))
    assert _rel(S_A + S_B, S_AB) > 0.1


def test_tab2_retnet_naive_addition_error():
    """Tab. 2 printed values: constant decay gamma and no write on C2 (beta = 0)
    make T_{C2} = gamma^{|C2|} I, so ||Delta|| / ||S_{C1|0}|| = 1 - gamma^{|C2|}."""
    path = os.path.join(os.path.dirname(__file__), "golden", "tab2_retnet_naive_addition.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    rng = _rng(13)
    d = 16
    C1 = _tokens(rng, 48, d, d)
    _, S_C1 = oracle.recurrence(*C1)
    checked = 0
    for e, n, printed in rows:
        gamma = 1.0 - 2.0 ** int(e)
        n = int(n)
        q2, k2, v2, _, _ = _tokens(rng, n, d, d)
        beta2 = np.zeros(n)
        a2 = np.full(n, np.log(gamma))
        P2, g2 = oracle.segment_operator(k2, beta2, a2)
        _, S_C2 = oracle.recurrence(q2, k2, v2, beta2, a2)
        S_true, _ = oracle.compose(P2[None, None], np.array([[g2]]), S_C2[None, None],
                                   [0], [0, 1], S_prefix=S_C1[None, None])
        delta = S_true[0, 0] - (S_C1 + S_C2)
        ratio = np.linalg.norm(delta) / np.linalg.norm(S_C1)
        assert f"{ratio:.3f}" == printed, (e, n, ratio, printed)
        checked += 1
    assert checked == 9


# --------------------------------------------------------------------------
# Batched build: segment independence, grouped heads
# --------------------------------------------------------------------------

def test_segment_alone_equals_segment_in_batch():
    rng = _rng(14)
    lens = [7, 64, 1, 30]
    q, k, v, beta, a, cu = _ragged_case(rng, lens, 6, 5, h_qk=2, h_v=4)
    out = oracle.build_segments(q, k, v, beta, a, cu)
    j = 1
    lo, hi = cu[j], cu[j + 1]
    alone = oracle.build_segments(q[lo:hi], k[lo:hi], v[lo:hi], beta[lo:hi], a[lo:hi],
                                  [0, hi - lo])
    assert np.array_equal(alone["S_seg"][0], out["S_seg"][j])
    assert np.array_equal(alone["P_hat"][0], out["P_hat"][j])
    assert np.array_equal(alone["o"], out["o"][lo:hi])


def test_grouped_heads_share_keys():
    """v-heads of one group read the same qk-head; with equal gates their
    operators coincide, with different values their states differ."""
    rng = _rng(15)
    lens = [20]
    q, k, v, beta, a, cu = _ragged_case(rng, lens, 6, 6, h_qk=2, h_v=4)
    beta[:, 1] = beta[:, 0]
    a[:, 1] = a[:, 0]
    out = oracle.build_segments(q, k, v, beta, a, cu)
    assert np.array_equal(out["P_hat"][0, 0], out["P_hat"][0, 1])
    assert out["log_decay"][0, 0] == out["log_decay"][0, 1]
    assert not np.allclose(out["S_seg"][0, 0], out["S_seg"][0, 1])
    # v-head 2 reads qk-head 1
    P2, _ = oracle.segment_operator(k[:, 1], beta[:, 2], a[:, 2])
    assert np.array_equal(out["P_hat"][0, 2], P2)
    assert gdn.qk_head_of(3, 4, 2) == 1 and gdn.qk_head_of(1, 4, 2) == 0


def test_seam_longer_than_segment_uses_whole_segment():
    rng = _rng(16)
    lens = [3, 12]
    q, k, v, beta, a, cu = _ragged_case(rng, lens, 5, 4)
    S_in = rng.standard_normal((2, 1, 5, 4))
    o_seam, S_post = oracle.seam(q, k, v, beta, a, cu[:-1], lens, 8, S_in)
    o_ref, S_ref = oracle.recurrence(q[:3, 0], k[:3, 0], v[:3, 0], beta[:3, 0], a[:3, 0],
                                     S0=S_in[0, 0])
    assert np.array_equal(o_seam[0, :3, 0], o_ref)
    assert np.all(np.isnan(o_seam[0, 3:, 0]))
    assert np.array_equal(S_post[0, 0], S_ref)


# --------------------------------------------------------------------------
# Sensitivity: mistakes planted in a copy of the oracle's recurrence fail the
# brute-force pin above (the planted copies live only in this test).
# --------------------------------------------------------------------------

def _mutant(kind):
    def rec(q, k, v, beta, a, S0=None):
        L, d_k = k.shape
        S = np.zeros((d_k, v.shape[1])) if S0 is None else S0.copy()
        o = np.zeros((L, v.shape[1]))
        for t in range(L):
            S_prev = S
            sign = 1.0 if kind == "sign" else -1.0
            S = np.exp(a[t]) * (S + sign * beta[t] * np.outer(k[t], k[t] @ S))
            if kind == "gate_on_write":
                S = S + np.exp(a[t]) * beta[t] * np.outer(k[t], v[t])
            else:
                S = S + beta[t] * np.outer(k[t], v[t])
            o[t] = (S_prev if kind == "read_before_write" else S).T @ q[t]
        return o, S
    return rec


@pytest.mark.parametrize("kind", ["sign", "gate_on_write", "read_before_write"])
def test_planted_mistakes_are_caught(kind):
    rng = _rng(17)
    L, d_k, d_v = 12, 6, 5
    q, k, v, beta, a = _tokens(rng, L, d_k, d_v, a_range=(-0.5, -0.1))
    T = _factors(k, beta, a)
    o_ref = np.zeros((L, d_v))
    S_t = np.zeros((d_k, d_v))
    for t in range(L):
        S_t = T[t] @ S_t + beta[t] * np.outer(k[t], v[t])
        o_ref[t] = q[t] @ S_t
    o_good, _ = oracle.recurrence(q, k, v, beta, a)
    o_bad, _ = _mutant(kind)(q, k, v, beta, a)
    assert _rel(o_good, o_ref) < 1e-12
    assert _rel(o_bad, o_ref) > 1e-3


# --------------------------------------------------------------------------
# Seam windows that advance the state (Sec. 4.3, reading A)
# --------------------------------------------------------------------------

def test_seam_advance_reuse_equals_concatenated_recurrence():
    """Entries cached as tail tuples over [w, L) and reused with their seams run
    from the composed state reproduce, for each request, the recurrence over the
    concatenation of its segments behind the prefix: the end state, and the
    outputs at every seam position (including a segment shorter than w)."""
    rng = np.random.default_rng(91)
    d_k, d_v, h_qk, h_v, w = 6, 5, 1, 2, 4
    lens = [9, 3, 12, 7]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    q = rng.standard_normal((T, h_qk, d_k))
    k = rng.standard_normal((T, h_qk, d_k))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, h_v, d_v))
    beta = rng.uniform(0.1, 0.9, size=(T, h_v))
    la = rng.uniform(-0.2, 0.0, size=(T, h_v))
    # tail tuples: tokens [start + w_i, end) of each entry
    tails = [(int(cu[i]) + min(w, lens[i]), int(cu[i + 1])) for i in range(4)]
    P = np.zeros((4, h_v, d_k, d_k))
    ld = np.zeros((4, h_v))
    S = np.zeros((4, h_v, d_k, d_v))
    for i, (a, b) in enumerate(tails):
        for h in range(h_v):
            _, S[i, h] = gdn.recurrence(q[a:b, 0], k[a:b, 0], v[a:b, h], beta[a:b, h], la[a:b, h])
            P[i, h], ld[i, h] = gdn.segment_operator(k[a:b, 0], beta[a:b, h], la[a:b, h])
    ids = [2, 0, 1, 3, 1]
    offs = [0, 3, 5]
    prefix = rng.standard_normal((2, h_v, d_k, d_v))
    S_out, o_seam, S_inc = gdn.compose_with_seams(P, ld, S, q, k, v, beta, la, cu[:-1], lens, w,
                                                  ids, offs, S_prefix=prefix)
    for r in range(2):
        sel = ids[offs[r]:offs[r + 1]]
        idx = np.concatenate([np.arange(cu[i], cu[i + 1]) for i in sel])
        for h in range(h_v):
            o_full, S_full = gdn.recurrence(q[idx, 0], k[idx, 0], v[idx, h], beta[idx, h],
                                            la[idx, h], S0=prefix[r, h])
            assert np.allclose(S_out[r, h], S_full, atol=1e-12, rtol=0)
            pos = 0
            for j, i in enumerate(sel):
                wi = min(w, lens[i])
                jj = offs[r] + j
                assert np.allclose(o_seam[jj, :wi, h], o_full[pos:pos + wi], atol=1e-12, rtol=0)
                assert np.all(np.isnan(o_seam[jj, wi:, h]))
                pos += lens[i]
    # the incoming state of the first listed entry is the prefix
    assert np.array_equal(S_inc[0], prefix[0])


def test_seam_advance_differs_from_full_tuples_plus_advancing_seam():
    """Applying the full-segment tuple after a seam that already advanced the
    state counts the seam tokens twice: the result is wrong, so the tuple must be
    the tail's (a planted-mistake check on the reading)."""
    rng = np.random.default_rng(92)
    d, L, w = 5, 10, 4
    q, k, v = (rng.standard_normal((L, 1, d)) for _ in range(3))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    beta = rng.uniform(0.2, 0.9, size=(L, 1))
    la = rng.uniform(-0.2, 0.0, size=(L, 1))
    _, S_full_tuple = gdn.recurrence(q[:, 0], k[:, 0], v[:, 0], beta[:, 0], la[:, 0])
    P_full, ld_full = gdn.segment_operator(k[:, 0], beta[:, 0], la[:, 0])
    prefix = rng.standard_normal((1, 1, d, d))
    wrong, _, _ = gdn.compose_with_seams(P_full[None, None], np.array([[ld_full]]),
                                         S_full_tuple[None, None], q, k, v, beta, la, [0], [L],
                                         w, [0], [0, 1], S_prefix=prefix)
    _, right = gdn.recurrence(q[:, 0], k[:, 0], v[:, 0], beta[:, 0], la[:, 0], S0=prefix[0, 0])
    assert np.linalg.norm(wrong[0, 0] - right) / np.linalg.norm(right) > 1e-3
