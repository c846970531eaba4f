"""Float64 oracle for the other transition families of Tab. 1 and the adjacent
reuse-time steps of Sec. 4.2 (conv warm-up, state RoPE shift, Eq. (7)) and
Sec. 4.3 (cached-key re-rotation, Eq. (8)).

TEST INFRASTRUCTURE ONLY (see the package docstring): this module defines what
the HIP path must reproduce and is never used by it.

Families, per head and token t (Tab. 1; the write has no beta for these rows):

* scalar (RetNet, Lightning-2, Mamba2): ``T_t = exp(a_t) I`` with one gate
  ``a_t`` per (token, head) (RetNet's constant decay is ``a_t = log gamma``);
* diagonal (GLA): ``T_t = diag(exp(g_t))`` with a gate vector ``g_t`` in
  R^{d_k} per (token, head);

with ``u_t = k_t v_t^T`` and Eq. (2): ``S_t = T_t S_{t-1} + u_t``,
``o_t = S_t^T q_t``.  Tab. 3 stores their segment operators compressed: a
scalar ``prod_t exp(a_t)`` and a vector ``prod_t exp(g_t)``; here both are
carried as logarithms (``log_decay = sum_t a_t`` or ``sum_t g_t``), which do not
underflow on long segments.

RoPE (Eq. (7), Eq. (8)): ``R(p)`` rotates channel pairs (2i, 2i+1) by the angle
``p * theta_i`` with ``theta_i = base^(-2i/d)``, the pairing of the RoPE paper
the text cites (the paper does not fix a pairing).

Conv warm-up (Sec. 4.2): a depthwise causal convolution of width K over the
hidden channels, ``y[t, c] = silu(sum_j w[c, j] x[t - K + 1 + j, c])``, whose
first K - 1 inputs of a window come from the conv state (the K - 1 raw inputs
that precede it; zero for a segment cached on its own).

All arithmetic is numpy float64; inputs are upcast exactly.
"""

import numpy as np

from .gdn import qk_head_of

SCALAR = "scalar"
DIAGONAL = "diagonal"


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def family_recurrence(family, q, k, v, gate, S0=None):
    """Eq. (2) over one head for the scalar or diagonal family of Tab. 1.

    q, k: [L, d_k]; v: [L, d_v]; gate: [L] (scalar: a_t) or [L, d_k]
    (diagonal: g_t), natural-log units; S0: [d_k, d_v] or None (zero start).
    For each token, in order:

        scalar:   S <- exp(a_t) S + k_t v_t^T
        diagonal: S <- diag(exp(g_t)) S + k_t v_t^T
        o_t = S^T q_t

    Returns (o [L, d_v], S_end [d_k, d_v]).
    """
    q, k, v, gate = _f64(q), _f64(k), _f64(v), _f64(gate)
    L, d_k = k.shape
    d_v = v.shape[1]
    S = np.zeros((d_k, d_v)) if S0 is None else np.array(S0, dtype=np.float64)
    o = np.zeros((L, d_v))
    for t in range(L):
        if family == SCALAR:
            S = np.exp(gate[t]) * S
        elif family == DIAGONAL:
            S = np.exp(gate[t])[:, None] * S
        else:
            raise ValueError(family)
        S = S + np.outer(k[t], v[t])
        o[t] = S.T @ q[t]
    return o, S


def family_log_decay(family, gate):
    """Logarithm of the compressed segment operator of Tab. 3: the sum over the
    segment's tokens of a_t (scalar, a float) or of g_t (diagonal, [d_k])."""
    gate = _f64(gate)
    if family == SCALAR:
        return float(np.sum(gate))
    return np.sum(gate, axis=0)


def _gate_slice(gate, lo, hi, h):
    return gate[lo:hi, h] if gate.ndim == 2 else gate[lo:hi, h, :]


def family_build_segments(family, q, k, v, gate, cu_seqlens, seg_head_pairs=None):
    """Zero-start build of every segment of a packed batch (Sec. 4.2 cache tuple
    with the Tab. 3 compressed operator).

    q, k: [T, h_qk, d_k]; v: [T, h_v, d_v]; gate: [T, h_v] (scalar) or
    [T, h_v, d_k] (diagonal).  Returns dict with o [T, h_v, d_v],
    S_seg [n_seg, h_v, d_k, d_v] and log_decay [n_seg, h_v] (scalar) or
    [n_seg, h_v, d_k] (diagonal); pairs not listed stay NaN.
    """
    gate = _f64(gate)
    T, h_qk, d_k = np.shape(k)
    h_v, d_v = np.shape(v)[1], np.shape(v)[2]
    cu = [int(x) for x in cu_seqlens]
    n_seg = len(cu) - 1
    o = np.full((T, h_v, d_v), np.nan)
    S_seg = np.full((n_seg, h_v, d_k, d_v), np.nan)
    ld_shape = (n_seg, h_v) if family == SCALAR else (n_seg, h_v, d_k)
    log_decay = np.full(ld_shape, np.nan)
    if seg_head_pairs is None:
        seg_head_pairs = [(s, h) for s in range(n_seg) for h in range(h_v)]
    for s, h in seg_head_pairs:
        lo, hi = cu[s], cu[s + 1]
        g = qk_head_of(h, h_v, h_qk)
        gs = _gate_slice(gate, lo, hi, h)
        o[lo:hi, h], S_seg[s, h] = family_recurrence(family, q[lo:hi, g], k[lo:hi, g],
                                                     v[lo:hi, h], gs)
        log_decay[s, h] = family_log_decay(family, gs) if hi > lo else 0.0
    return {"o": o, "S_seg": S_seg, "log_decay": log_decay}


def family_compose(family, log_decay, S_seg, seg_ids, req_offsets, S_prefix=None,
                   req_head_pairs=None):
    """Eq. (6) with the compressed operators of Tab. 3, as repeated Eq. (4):
    each listed segment i maps the running state S to ``T_i S + S_i`` with
    ``T_i = exp(log_decay_i) I`` (scalar) or ``diag(exp(log_decay_i))``
    (diagonal).  Returns (S_out [n_req, h_v, d_k, d_v], S_incoming [nnz, ...]),
    S_incoming[j] being the state just before listed segment j."""
    S_seg = np.asarray(S_seg)
    log_decay = _f64(log_decay)
    n_pool, h_v, d_k, d_v = S_seg.shape
    offs = [int(x) for x in req_offsets]
    ids = [int(x) for x in seg_ids]
    n_req = len(offs) - 1
    S_out = np.full((n_req, h_v, d_k, d_v), np.nan)
    S_inc = np.full((len(ids), h_v, d_k, d_v), np.nan)
    if req_head_pairs is None:
        req_head_pairs = [(r, h) for r in range(n_req) for h in range(h_v)]
    for r, h in req_head_pairs:
        S = np.zeros((d_k, d_v)) if S_prefix is None else _f64(S_prefix[r, h]).copy()
        for j in range(offs[r], offs[r + 1]):
            i = ids[j]
            S_inc[j, h] = S
            if family == SCALAR:
                T_i = np.exp(log_decay[i, h]) * np.eye(d_k)
            else:
                T_i = np.diag(np.exp(log_decay[i, h]))
            S = T_i @ S + _f64(S_seg[i, h])
        S_out[r, h] = S
    return S_out, S_inc


def family_seam(family, q, k, v, gate, tok_start, tok_len, w, S_in, entry_head_pairs=None):
    """Seam rescan (Sec. 4.3) for the scalar or diagonal family: the first
    ``min(w, tok_len[e])`` tokens of entry e run through Eq. (2) from S_in[e].
    Returns (o_seam [n, w, h_v, d_v] with rows past w_eff NaN, S_post)."""
    gate = _f64(gate)
    T, h_qk, d_k = np.shape(k)
    h_v, d_v = np.shape(v)[1], np.shape(v)[2]
    n_e = len(tok_start)
    o_seam = np.full((n_e, w, h_v, d_v), np.nan)
    S_post = np.full((n_e, h_v, d_k, d_v), np.nan)
    if entry_head_pairs is None:
        entry_head_pairs = [(e, h) for e in range(n_e) for h in range(h_v)]
    for e, h in entry_head_pairs:
        lo = int(tok_start[e])
        hi = lo + min(int(w), int(tok_len[e]))
        g = qk_head_of(h, h_v, h_qk)
        o_eh, S_eh = family_recurrence(family, q[lo:hi, g], k[lo:hi, g], v[lo:hi, h],
                                       _gate_slice(gate, lo, hi, h), S0=S_in[e, h])
        o_seam[e, :hi - lo, h] = o_eh
        S_post[e, h] = S_eh
    return o_seam, S_post


# ---------------------------------------------------------------------------
# RoPE: Eq. (7) state shift and Eq. (8) key re-rotation
# ---------------------------------------------------------------------------

def rope_angles(d, base):
    """theta_i = base^(-2i/d) for the d/2 channel pairs."""
    i = np.arange(d // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * i / d)


def rope_matrix(p, d, base):
    """R(p): block-diagonal rotation of channel pairs (2i, 2i+1) by p * theta_i,
    built entry by entry."""
    th = rope_angles(d, base)
    R = np.zeros((d, d))
    for i in range(d // 2):
        c, s = np.cos(p * th[i]), np.sin(p * th[i])
        R[2 * i, 2 * i] = c
        R[2 * i, 2 * i + 1] = -s
        R[2 * i + 1, 2 * i] = s
        R[2 * i + 1, 2 * i + 1] = c
    return R


def rope_shift_state(S, delta, base):
    """Eq. (7): the state of a scalar-family segment moved by ``delta``
    positions, ``R(delta) S`` (S: [d_k, d_v])."""
    S = _f64(S)
    return rope_matrix(delta, S.shape[0], base) @ S


def rope_rerotate_keys(K, delta, base):
    """Eq. (8): cached keys moved by ``delta`` positions, ``K_b = R(delta) K_a``
    applied to every key (rows of K: [L, d_k])."""
    K = _f64(K)
    return K @ rope_matrix(delta, K.shape[1], base).T


def rope_keys_at(K, start, base):
    """Keys of consecutive tokens rotated to absolute positions start, start+1, ..."""
    K = _f64(K)
    return np.stack([rope_matrix(start + t, K.shape[1], base) @ K[t]
                     for t in range(K.shape[0])]) if len(K) else K.copy()


# ---------------------------------------------------------------------------
# causal conv warm-up (Sec. 4.2)
# ---------------------------------------------------------------------------

def silu(x):
    return x / (1.0 + np.exp(-x))


def causal_conv(x, weight, conv_state=None, activation=True):
    """Depthwise causal convolution of one window of raw inputs.

    x: [L, C]; weight: [C, K]; conv_state: [K - 1, C] raw inputs that precede
    the window (zero when None).  y[t, c] = silu(sum_j weight[c, j] *
    xx[t + j, c]) over xx = concat(conv_state, x).  Returns (y [L, C], the
    trailing conv state [K - 1, C]: the last K - 1 rows of xx).
    """
    x, weight = _f64(x), _f64(weight)
    L, C = x.shape
    K = weight.shape[1]
    st = np.zeros((K - 1, C)) if conv_state is None else _f64(conv_state)
    xx = np.concatenate([st, x], axis=0)
    y = np.zeros((L, C))
    for t in range(L):
        for j in range(K):
            y[t] += weight[:, j] * xx[t + j]
    if activation:
        y = silu(y)
    return y, xx[L:].copy() if K > 1 else np.zeros((0, C))
