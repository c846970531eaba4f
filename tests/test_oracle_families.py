"""Pins of the float64 oracle for the scalar and diagonal families of Tab. 1,
the RoPE state shift (Eq. (7)) and key re-rotation (Eq. (8)), and the causal
conv warm-up (Sec. 4.2).

Each check is computed independently of the oracle's code path: explicit factor
matrices, closed forms, the printed Tab. 2 values, library routines
(np.convolve) and brute force.  CPU only.
"""

import os

import numpy as np
import pytest

from oracle import families as F
from oracle import gdn


def _rng(seed):
    return np.random.default_rng(seed)


def _rel(x, ref):
    return np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-300)


def _tokens(rng, L, d_k, d_v, family, g_range=(-0.3, 0.0)):
    q = rng.standard_normal((L, d_k))
    k = rng.standard_normal((L, d_k))
    v = rng.standard_normal((L, d_v))
    shape = (L,) if family == F.SCALAR else (L, d_k)
    gate = rng.uniform(*g_range, size=shape)
    return q, k, v, gate


def _transition(family, gate_t, d_k):
    """Explicit T_t of Tab. 1 as a d_k x d_k matrix."""
    if family == F.SCALAR:
        return np.exp(gate_t) * np.eye(d_k)
    return np.diag(np.exp(gate_t))


def _left_product(mats, d):
    P = np.eye(d)
    for M in mats:
        P = M @ P
    return P


# --------------------------------------------------------------------------
# Brute force of Eq. (2) with explicit factor matrices
# --------------------------------------------------------------------------

@pytest.mark.parametrize("family", [F.SCALAR, F.DIAGONAL])
@pytest.mark.parametrize("with_s0", [False, True])
def test_family_recurrence_matches_explicit_factor_sums(family, with_s0):
    rng = _rng(31)
    L, d_k, d_v = 20, 8, 6
    q, k, v, gate = _tokens(rng, L, d_k, d_v, family, g_range=(-0.8, 0.2))
    S0 = rng.standard_normal((d_k, d_v)) if with_s0 else None
    T = [_transition(family, gate[t], d_k) for t in range(L)]
    u = [np.outer(k[t], v[t]) for t in range(L)]
    o_ref = np.zeros((L, d_v))
    for t in range(L):
        S_t = np.zeros((d_k, d_v)) if S0 is None else _left_product(T[:t + 1], d_k) @ S0
        for s in range(t + 1):
            S_t = S_t + _left_product(T[s + 1:t + 1], d_k) @ u[s]
        o_ref[t] = q[t] @ S_t
    o, S = F.family_recurrence(family, q, k, v, gate, S0=S0)
    assert _rel(o, o_ref) < 1e-12
    assert _rel(S, S_t) < 1e-12
    # Tab. 3 compressed operator: the ordered product of the T_t
    T_C = _left_product(T, d_k)
    ld = F.family_log_decay(family, gate)
    T_ld = np.exp(ld) * np.eye(d_k) if family == F.SCALAR else np.diag(np.exp(ld))
    assert _rel(T_ld, T_C) < 1e-12


def test_scalar_constant_decay_closed_form():
    """RetNet row: S_L = sum_t gamma^(L-1-t) k_t v_t^T, T_C = gamma^L I."""
    rng = _rng(32)
    L, d_k, d_v = 30, 7, 5
    gamma = 0.93
    q, k, v, _ = _tokens(rng, L, d_k, d_v, F.SCALAR)
    S_ref = sum(gamma ** (L - 1 - t) * np.outer(k[t], v[t]) for t in range(L))
    o, S = F.family_recurrence(F.SCALAR, q, k, v, np.full(L, np.log(gamma)))
    assert _rel(S, S_ref) < 1e-12
    assert abs(F.family_log_decay(F.SCALAR, np.full(L, np.log(gamma))) - L * np.log(gamma)) < 1e-12


def test_diagonal_basis_key_closed_form():
    """Every key equal to basis vector e_c: S = e_c s^T with the scalar
    recurrence s_t = exp(g_t[c]) s_{t-1} + v_t on that channel only."""
    rng = _rng(33)
    L, d_k, d_v, c = 25, 6, 4, 3
    _, _, v, gate = _tokens(rng, L, d_k, d_v, F.DIAGONAL)
    k = np.zeros((L, d_k))
    k[:, c] = 1.0
    q = rng.standard_normal((L, d_k))
    s = np.zeros(d_v)
    for t in range(L):
        s = np.exp(gate[t, c]) * s + v[t]
    _, S = F.family_recurrence(F.DIAGONAL, q, k, v, gate)
    S_ref = np.zeros((d_k, d_v))
    S_ref[c] = s
    assert _rel(S, S_ref) < 1e-12


def test_diagonal_with_uniform_gates_is_scalar():
    rng = _rng(34)
    L, d_k, d_v = 18, 6, 5
    q, k, v, a = _tokens(rng, L, d_k, d_v, F.SCALAR)
    o1, S1 = F.family_recurrence(F.SCALAR, q, k, v, a)
    o2, S2 = F.family_recurrence(F.DIAGONAL, q, k, v, np.repeat(a[:, None], d_k, axis=1))
    assert _rel(o2, o1) < 1e-14 and _rel(S2, S1) < 1e-14


def test_diagonal_zero_write_pure_decay():
    rng = _rng(35)
    L, d_k, d_v = 10, 5, 3
    q, _, _, gate = _tokens(rng, L, d_k, d_v, F.DIAGONAL)
    S0 = rng.standard_normal((d_k, d_v))
    _, S = F.family_recurrence(F.DIAGONAL, q, np.zeros((L, d_k)), np.zeros((L, d_v)), gate, S0=S0)
    assert _rel(S, np.exp(gate.sum(axis=0))[:, None] * S0) < 1e-12


# --------------------------------------------------------------------------
# Composition (Eq. 4 / Eq. 6) and seams against the concatenated run
# --------------------------------------------------------------------------

def _packed(rng, family, lens, d_k, d_v, h_qk, h_v, g_range=(-0.1, 0.0)):
    T = sum(lens)
    q = rng.standard_normal((T, h_qk, d_k))
    k = rng.standard_normal((T, h_qk, d_k))
    v = rng.standard_normal((T, h_v, d_v))
    shape = (T, h_v) if family == F.SCALAR else (T, h_v, d_k)
    gate = rng.uniform(*g_range, size=shape)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return q, k, v, gate, cu


@pytest.mark.parametrize("family", [F.SCALAR, F.DIAGONAL])
def test_family_compose_behind_prefix_equals_concatenation_and_seams(family):
    rng = _rng(36)
    lens = [9, 14, 1, 20]
    d_k, d_v, h_qk, h_v = 6, 5, 1, 2
    q, k, v, gate, cu = _packed(rng, family, lens, d_k, d_v, h_qk, h_v, g_range=(-0.4, 0.1))
    S_prefix = rng.standard_normal((1, h_v, d_k, d_v))
    built = F.family_build_segments(family, q, k, v, gate, cu)
    ids = np.arange(len(lens))
    S_out, S_inc = F.family_compose(family, built["log_decay"], built["S_seg"], ids,
                                    [0, len(lens)], S_prefix=S_prefix)
    w = 4
    o_seam, S_post = F.family_seam(family, q, k, v, gate, cu[:-1], np.diff(cu), w, S_inc)
    for h in range(h_v):
        g = gdn.qk_head_of(h, h_v, h_qk)
        gh = gate[:, h]
        o_full, S_full = F.family_recurrence(family, q[:, g], k[:, g], v[:, h], gh,
                                             S0=S_prefix[0, h])
        assert _rel(S_out[0, h], S_full) < 1e-12
        for j, s in enumerate(ids):
            lo = int(cu[s])
            we = min(w, lens[s])
            # the incoming state is the full run's state just before the segment
            _, S_before = F.family_recurrence(family, q[:lo, g], k[:lo, g], v[:lo, h], gh[:lo],
                                              S0=S_prefix[0, h])
            assert _rel(S_inc[j, h], S_before) < 1e-12
            assert _rel(o_seam[j, :we, h], o_full[lo:lo + we]) < 1e-12


@pytest.mark.parametrize("family", [F.SCALAR, F.DIAGONAL])
def test_family_compose_literal_eq6_sum(family):
    """Eq. (6) written term by term, with the compressed operators."""
    rng = _rng(37)
    n, d_k, d_v = 4, 5, 3
    S_seg = rng.standard_normal((n, 1, d_k, d_v))
    shape = (n, 1) if family == F.SCALAR else (n, 1, d_k)
    ld = rng.uniform(-2.0, 0.5, size=shape)
    S_pre = rng.standard_normal((d_k, d_v))
    order = [2, 0, 3, 1]
    T = [_transition(family, ld[i, 0], d_k) for i in order]
    ref = _left_product(T, d_k) @ S_pre
    for i in range(n):
        ref = ref + _left_product(T[i + 1:], d_k) @ S_seg[order[i], 0]
    S_out, _ = F.family_compose(family, ld, S_seg, order, [0, n], S_prefix=S_pre[None, None])
    assert _rel(S_out[0, 0], ref) < 1e-13


@pytest.mark.parametrize("family", [F.SCALAR, F.DIAGONAL])
def test_family_naive_addition_fails(family):
    rng = _rng(38)
    d = 8
    A = _tokens(rng, 40, d, d, family, g_range=(-0.05, -0.01))
    B = _tokens(rng, 40, d, d, family, g_range=(-0.05, -0.01))
    _, S_A = F.family_recurrence(family, *A)
    _, S_B = F.family_recurrence(family, *B)
    cat = [np.concatenate([x, y]) for x, y in zip(A, B)]
    _, S_AB = F.family_recurrence(family, *cat)
    assert _rel(S_A + S_B, S_AB) > 0.1


def test_tab2_printed_values_through_scalar_compose():
    """Tab. 2 (RetNet, T_t = gamma I): ||Delta|| / ||S_{C1|0}|| = 1 - gamma^{|C2|}
    for the naive sum against the Eq. (6) composition with the scalar operator."""
    path = os.path.join(os.path.dirname(__file__), "golden", "tab2_retnet_naive_addition.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    rng = _rng(39)
    d = 12
    C1 = _tokens(rng, 40, d, d, F.SCALAR)
    _, S_C1 = F.family_recurrence(F.SCALAR, *C1)
    for e, n, printed in rows:
        gamma = 1.0 - 2.0 ** int(e)
        n = int(n)
        q2, k2, v2, _ = _tokens(rng, n, d, d, F.SCALAR)
        a2 = np.full(n, np.log(gamma))
        _, S_C2 = F.family_recurrence(F.SCALAR, q2, k2, v2, a2)
        ld = np.array([[F.family_log_decay(F.SCALAR, a2)]])
        S_true, _ = F.family_compose(F.SCALAR, ld, S_C2[None, None], [0], [0, 1],
                                     S_prefix=S_C1[None, None])
        ratio = np.linalg.norm(S_true[0, 0] - (S_C1 + S_C2)) / np.linalg.norm(S_C1)
        assert f"{ratio:.3f}" == printed, (e, n, ratio, printed)


def _family_mutant(kind):
    def rec(q, k, v, gate, S0=None):
        L, d_k = k.shape
        S = np.zeros((d_k, v.shape[1])) if S0 is None else S0.copy()
        o = np.zeros((L, v.shape[1]))
        for t in range(L):
            if kind == "gate_on_columns":
                S = S * np.exp(gate[t])[None, :]
            else:
                S = np.exp(gate[t])[:, None] * S
            w = np.outer(k[t], v[t])
            S = S + (np.exp(gate[t])[:, None] * w if kind == "gate_on_write" else w)
            o[t] = S.T @ q[t]
        return o, S
    return rec


@pytest.mark.parametrize("kind", ["gate_on_columns", "gate_on_write"])
def test_family_planted_mistakes_are_caught(kind):
    rng = _rng(40)
    L, d = 10, 6   # d_k == d_v so that the column-gated copy runs
    q, k, v, gate = _tokens(rng, L, d, d, F.DIAGONAL, g_range=(-0.6, -0.1))
    S_t = np.zeros((d, d))
    o_ref = np.zeros((L, d))
    for t in range(L):
        S_t = np.diag(np.exp(gate[t])) @ S_t + np.outer(k[t], v[t])
        o_ref[t] = q[t] @ S_t
    o_good, _ = F.family_recurrence(F.DIAGONAL, q, k, v, gate)
    o_bad, _ = _family_mutant(kind)(q, k, v, gate)
    assert _rel(o_good, o_ref) < 1e-12
    assert _rel(o_bad, o_ref) > 1e-3


# --------------------------------------------------------------------------
# RoPE: Eq. (7) and Eq. (8)
# --------------------------------------------------------------------------

def test_rope_is_a_rotation_group():
    d, base = 16, 10000.0
    I = np.eye(d)
    assert np.allclose(F.rope_matrix(0, d, base), I, atol=0, rtol=0)
    for a, b in [(3, 5), (-7, 100), (1000, 24)]:
        Ra, Rb, Rab = (F.rope_matrix(x, d, base) for x in (a, b, a + b))
        assert np.allclose(Ra @ Rb, Rab, atol=1e-12)
        assert np.allclose(Ra.T @ Ra, I, atol=1e-13)
    # relative-position property of RoPE scores: (R(m) q) . (R(n) k) depends on m - n
    rng = _rng(41)
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    s1 = (F.rope_matrix(30, d, base) @ q) @ (F.rope_matrix(12, d, base) @ k)
    s2 = (F.rope_matrix(118, d, base) @ q) @ (F.rope_matrix(100, d, base) @ k)
    assert abs(s1 - s2) < 1e-12


def test_rope_pairs_rotate_by_their_own_angle():
    """Each 2 x 2 block acts on channels (2i, 2i+1) only, as a rotation by
    p * base^(-2i/d); other blocks are zero."""
    d, base, p = 8, 500.0, 7
    R = F.rope_matrix(p, d, base)
    for i in range(d // 2):
        blk = R[2 * i:2 * i + 2, 2 * i:2 * i + 2]
        ang = np.arctan2(blk[1, 0], blk[0, 0])
        want = (p * base ** (-2.0 * i / d) + np.pi) % (2 * np.pi) - np.pi
        assert abs(ang - want) < 1e-12
        off = R[2 * i:2 * i + 2].copy()
        off[:, 2 * i:2 * i + 2] = 0
        assert np.all(off == 0)


def test_eq7_state_shift_holds_for_scalar_family():
    """A scalar-family segment whose keys carry RoPE at absolute positions
    a, a+1, ... has S_{C|b} = R(b - a) S_{C|a} (Eq. 7)."""
    rng = _rng(42)
    L, d_k, d_v, base = 24, 8, 5, 10000.0
    q, k, v, a = _tokens(rng, L, d_k, d_v, F.SCALAR)
    pa, pb = 5, 321
    _, S_a = F.family_recurrence(F.SCALAR, q, F.rope_keys_at(k, pa, base), v, a)
    _, S_b = F.family_recurrence(F.SCALAR, q, F.rope_keys_at(k, pb, base), v, a)
    assert _rel(F.rope_shift_state(S_a, pb - pa, base), S_b) < 1e-12
    # it is not an identity of the test: per-channel (diagonal) gates that differ
    # within a rotated pair do not commute with R ...
    g = rng.uniform(-0.3, 0.0, size=(L, d_k))
    _, D_a = F.family_recurrence(F.DIAGONAL, q, F.rope_keys_at(k, pa, base), v, g)
    _, D_b = F.family_recurrence(F.DIAGONAL, q, F.rope_keys_at(k, pb, base), v, g)
    assert _rel(F.rope_shift_state(D_a, pb - pa, base), D_b) > 1e-3
    # ... while gates shared by the two channels of each pair do
    g2 = np.repeat(g[:, ::2], 2, axis=1)
    _, D_a = F.family_recurrence(F.DIAGONAL, q, F.rope_keys_at(k, pa, base), v, g2)
    _, D_b = F.family_recurrence(F.DIAGONAL, q, F.rope_keys_at(k, pb, base), v, g2)
    assert _rel(F.rope_shift_state(D_a, pb - pa, base), D_b) < 1e-12


def test_eq7_reuse_composition_equals_rotated_concatenation():
    """Sec. 4.2 reuse: Eq. (6) with each S_{C_i|0} replaced by R(p_i) S_{C_i|0}
    equals the scalar-family run over the concatenation with keys at their
    global positions."""
    rng = _rng(43)
    lens, d_k, d_v, base = [7, 12, 5], 8, 4, 10000.0
    segs = [_tokens(rng, L, d_k, d_v, F.SCALAR) for L in lens]
    S_seg, ld, starts, p = [], [], [], 0
    for (q, k, v, a) in segs:
        _, S = F.family_recurrence(F.SCALAR, q, F.rope_keys_at(k, 0, base), v, a)
        S_seg.append(S)
        ld.append(F.family_log_decay(F.SCALAR, a))
        starts.append(p)
        p += len(a)
    shifted = np.stack([F.rope_shift_state(S, st, base) for S, st in zip(S_seg, starts)])
    S_out, _ = F.family_compose(F.SCALAR, np.array(ld)[:, None], shifted[:, None],
                                [0, 1, 2], [0, 3])
    q = np.concatenate([s[0] for s in segs])
    k = np.concatenate([s[1] for s in segs])
    v = np.concatenate([s[2] for s in segs])
    a = np.concatenate([s[3] for s in segs])
    _, S_full = F.family_recurrence(F.SCALAR, q, F.rope_keys_at(k, 0, base), v, a)
    assert _rel(S_out[0, 0], S_full) < 1e-12


def test_eq7_replacement_needs_a_commuting_operator():
    """For a dense (GDN) transition the shifted state alone is not enough: the
    cached operator built at position 0 does not commute with R, so Eq. (6) with
    R(p_i) S_{C_i|0} and the unshifted T_{C_i} misses the concatenated run."""
    rng = _rng(48)
    lens, d_k, d_v, base = [9, 11], 8, 4, 100.0
    segs = []
    for L in lens:
        q, k, v, a = _tokens(rng, L, d_k, d_v, F.SCALAR)
        k = k / np.linalg.norm(k, axis=1, keepdims=True)
        segs.append((q, k, v, rng.uniform(0.3, 1.0, size=L), a))
    P, ld, S_seg, starts, p = [], [], [], [], 0
    for (q, k, v, b, a) in segs:
        kr = F.rope_keys_at(k, 0, base)
        _, S = gdn.recurrence(q, kr, v, b, a)
        Ph, g = gdn.segment_operator(kr, b, a)
        P.append(Ph)
        ld.append(g)
        S_seg.append(F.rope_shift_state(S, p, base))
        starts.append(p)
        p += len(a)
    S_out, _ = gdn.compose(np.stack(P)[:, None], np.array(ld)[:, None],
                           np.stack(S_seg)[:, None], [0, 1], [0, 2])
    cat = [np.concatenate([s[i] for s in segs]) for i in range(5)]
    _, S_full = gdn.recurrence(cat[0], F.rope_keys_at(cat[1], 0, base), *cat[2:])
    assert _rel(S_out[0, 0], S_full) > 1e-3


def test_eq8_key_rerotation():
    rng = _rng(44)
    L, d, base = 9, 16, 10000.0
    k = rng.standard_normal((L, d))
    Ka = F.rope_keys_at(k, 40, base)
    Kb = F.rope_keys_at(k, 1017, base)
    assert _rel(F.rope_rerotate_keys(Ka, 1017 - 40, base), Kb) < 1e-12


# --------------------------------------------------------------------------
# Causal conv warm-up (Sec. 4.2, Sec. 4.3)
# --------------------------------------------------------------------------

def test_causal_conv_matches_numpy_convolve():
    rng = _rng(45)
    L, C, K = 13, 5, 4
    x = rng.standard_normal((L, C))
    w = rng.standard_normal((C, K))
    st = rng.standard_normal((K - 1, C))
    y, tail = F.causal_conv(x, w, conv_state=st, activation=False)
    xx = np.concatenate([st, x])
    for c in range(C):
        ref = np.convolve(xx[:, c], w[c, ::-1], mode="valid")
        assert np.allclose(y[:, c], ref, atol=1e-13, rtol=0)
    assert np.array_equal(tail, xx[-(K - 1):])
    ya, _ = F.causal_conv(x, w, conv_state=st)
    assert np.array_equal(ya, F.silu(y))  # the activation is applied to the conv output


def test_silu_identities():
    """SiLU pinned by properties its definition x sigmoid(x) implies, none of
    which restates it: silu(0) = 0; the odd part silu(x) - silu(-x) = x
    (because sigmoid(x) + sigmoid(-x) = 1); silu(x) -> x for large x and -> 0
    for large negative x; at x = ln 3, sigmoid = 3/4 exactly; the minimum
    near x = -1.2785 (where silu' = 0) has value -0.2784645...; a planted
    mistake (tanh in place of sigmoid) breaks the odd-part identity."""
    x = np.linspace(-30.0, 30.0, 6001)
    assert F.silu(np.array([0.0]))[0] == 0.0
    assert np.allclose(F.silu(x) - F.silu(-x), x, atol=1e-13, rtol=0)
    assert abs(F.silu(np.array([40.0]))[0] - 40.0) < 1e-15 * 40 + 1e-15
    assert abs(F.silu(np.array([-40.0]))[0]) < 1e-15
    assert abs(F.silu(np.array([np.log(3.0)]))[0] - 0.75 * np.log(3.0)) < 1e-15
    # the minimum of x sigmoid(x): silu' = 0 where 1 + x sigmoid(-x) = 0, i.e.
    # x* = -1 - W(1/e) (W the Lambert function) = -1.27846454276107..., and there
    # sigmoid(x*) = 1 + 1/x*, so silu(x*) = x* + 1
    xs = np.linspace(-1.4, -1.1, 300001)
    ys = F.silu(xs)
    assert abs(xs[np.argmin(ys)] - (-1.27846454276107)) < 2e-6
    assert abs(ys.min() - (-0.27846454276107)) < 1e-10
    wrong = x * np.tanh(x)
    assert not np.allclose(wrong - (-x) * np.tanh(-x), x, atol=1e-3)


def test_conv_state_carries_across_windows():
    """conv(x1 || x2) = conv(x1) then conv(x2) from x1's trailing state; with
    K = 1 the conv is pointwise."""
    rng = _rng(46)
    C, K = 6, 4
    x1, x2 = rng.standard_normal((11, C)), rng.standard_normal((2, C))
    w = rng.standard_normal((C, K))
    y12, t12 = F.causal_conv(np.concatenate([x1, x2]), w)
    y1, t1 = F.causal_conv(x1, w)
    y2, t2 = F.causal_conv(x2, w, conv_state=t1)
    assert np.allclose(np.concatenate([y1, y2]), y12, atol=1e-14, rtol=0)
    assert np.array_equal(t2, t12)      # a window shorter than K - 1 keeps older inputs
    w1 = rng.standard_normal((C, 1))
    y, _ = F.causal_conv(x1, w1)
    assert np.allclose(y, F.silu(x1 * w1[:, 0]), atol=1e-15, rtol=0)


def test_conv_warmup_repairs_only_the_first_k_minus_1_tokens():
    """A segment convolved on its own (zero conv state) differs from the
    concatenated run only in its first K - 1 outputs, which the reuse-time
    warm-up from the previous segment's trailing state restores."""
    rng = _rng(47)
    C, K = 4, 4
    xa, xb = rng.standard_normal((10, C)), rng.standard_normal((9, C))
    w = rng.standard_normal((C, K))
    y_cat, _ = F.causal_conv(np.concatenate([xa, xb]), w)
    y_b_alone, _ = F.causal_conv(xb, w)
    _, tail_a = F.causal_conv(xa, w)
    y_b_warm, _ = F.causal_conv(xb[:K - 1], w, conv_state=tail_a)
    ref_b = y_cat[len(xa):]
    assert np.allclose(y_b_alone[K - 1:], ref_b[K - 1:], atol=1e-14, rtol=0)
    assert not np.allclose(y_b_alone[:K - 1], ref_b[:K - 1])
    assert np.allclose(y_b_warm, ref_b[:K - 1], atol=1e-14, rtol=0)
