"""Float64 oracle for the KDA row of Tab. 1: the delta rule with a per-channel
(diagonal) gate, ``T_t = (I - beta_t k_t k_t^T) diag(exp(g_t))`` and
``u_t = beta_t k_t v_t^T``.

TEST INFRASTRUCTURE ONLY (see the package docstring): this module defines what
the HIP path must reproduce and is never used by it.

Per head and token t (Eq. (2) with the Tab. 1 KDA row):

    S_t = (I - beta_t k_t k_t^T) diag(exp(g_t)) S_{t-1} + beta_t k_t v_t^T
    o_t = S_t^T q_t

with the gate ``g_t`` in R^{d_k} in natural-log units.  Tab. 3 stores the
segment operator in full, ``T_C = prod_t (I - beta_t k_t k_t^T) diag(exp(g_t))``
(later tokens on the left).  Here it is carried as ``T_C = exp(log_decay) P_hat``
with a scalar ``log_decay`` that keeps ``P_hat`` in range on long segments.  The
oracle factors each token's gate by its largest channel, m_t = max_c g_tc:
``T_t = exp(m_t) (I - beta_t k_t k_t^T) diag(exp(g_t - m_t))``, so
``log_decay = sum_t m_t`` and ``P_hat`` is the product of the rescaled factors.
Tab. 3 fixes only ``T_C``; any scalar split gives the same operator, so a cache
may choose another one, and comparisons are made on ``T_C`` (the Eq. (6)
composition of the GDN tuples reads any split).

All arithmetic is numpy float64; inputs are upcast exactly.
"""

import numpy as np

from .gdn import qk_head_of


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def kda_recurrence(q, k, v, beta, gate, S0=None):
    """Eq. (2) with the KDA transition over one head.

    q, k: [L, d_k]; v: [L, d_v]; beta: [L]; gate: [L, d_k]; S0: [d_k, d_v] or
    None (zero start).  For each token, in order:

        S' = diag(exp(g_t)) S                  (the gate acts first, Tab. 1)
        S  = S' - beta_t k_t (k_t^T S') + beta_t k_t v_t^T
        o_t = S^T q_t

    Returns (o [L, d_v], S_end [d_k, d_v]).
    """
    q, k, v, beta, gate = _f64(q), _f64(k), _f64(v), _f64(beta), _f64(gate)
    L, d_k = k.shape
    d_v = v.shape[1]
    S = np.zeros((d_k, d_v)) if S0 is None else np.array(S0, dtype=np.float64)
    o = np.zeros((L, d_v))
    for t in range(L):
        kt = k[t]
        Sp = np.exp(gate[t])[:, None] * S
        S = Sp - beta[t] * np.outer(kt, kt @ Sp) + beta[t] * np.outer(kt, v[t])
        o[t] = S.T @ q[t]
    return o, S


def kda_transition_product(k, beta, gate):
    """``T_C`` of Tab. 3 for the KDA row: the same recurrence from ``S = I``
    with every write zeroed (the construction of Sec. 5), [d_k, d_k]."""
    k = _f64(k)
    L, d_k = k.shape
    _, T_C = kda_recurrence(np.zeros((L, d_k)), k, np.zeros((L, d_k)), beta, gate,
                            S0=np.eye(d_k))
    return T_C


def kda_operator(k, beta, gate):
    """``T_C`` of Tab. 3 as ``(log_decay, P_hat)`` with ``T_C = exp(log_decay) P_hat``:
    each token's factor is split as ``exp(m_t) (I - beta_t k_t k_t^T) diag(exp(g_t - m_t))``
    with ``m_t`` its largest gate, so ``P_hat`` is the ordered product of the
    rescaled factors (later tokens on the left) and ``log_decay = sum_t m_t``.
    k: [L, d_k]; beta: [L]; gate: [L, d_k]."""
    k, beta, gate = _f64(k), _f64(beta), _f64(gate)
    L, d_k = k.shape
    P = np.eye(d_k)
    ld = 0.0
    for t in range(L):
        m = float(np.max(gate[t]))
        Pp = np.exp(gate[t] - m)[:, None] * P
        P = Pp - beta[t] * np.outer(k[t], k[t] @ Pp)
        ld += m
    return ld, P


def kda_build_segments(q, k, v, beta, gate, cu_seqlens, want_operator=True,
                       seg_head_pairs=None):
    """Zero-start build of every segment of a packed batch (Sec. 4.2 cache tuple).

    q, k: [T, h_qk, d_k]; v: [T, h_v, d_v]; beta: [T, h_v]; gate: [T, h_v, d_k].
    Returns dict with o [T, h_v, d_v], S_seg [n_seg, h_v, d_k, d_v],
    P_hat [n_seg, h_v, d_k, d_k] and log_decay [n_seg, h_v] with
    ``T_C = exp(log_decay) P_hat`` in the split of ``kda_operator``; pairs not
    listed stay NaN.
    """
    T, h_qk, d_k = np.shape(k)
    h_v, d_v = np.shape(v)[1], np.shape(v)[2]
    cu = [int(x) for x in cu_seqlens]
    n_seg = len(cu) - 1
    o = np.full((T, h_v, d_v), np.nan)
    S_seg = np.full((n_seg, h_v, d_k, d_v), np.nan)
    P_hat = np.full((n_seg, h_v, d_k, d_k), np.nan) if want_operator else None
    log_decay = np.full((n_seg, h_v), np.nan) if want_operator else None
    if seg_head_pairs is None:
        seg_head_pairs = [(s, h) for s in range(n_seg) for h in range(h_v)]
    for s, h in seg_head_pairs:
        lo, hi = cu[s], cu[s + 1]
        g = qk_head_of(h, h_v, h_qk)
        o[lo:hi, h], S_seg[s, h] = kda_recurrence(q[lo:hi, g], k[lo:hi, g], v[lo:hi, h],
                                                  beta[lo:hi, h], gate[lo:hi, h])
        if want_operator:
            log_decay[s, h], P_hat[s, h] = kda_operator(k[lo:hi, g], beta[lo:hi, h],
                                                        gate[lo:hi, h])
    return {"o": o, "S_seg": S_seg, "P_hat": P_hat, "log_decay": log_decay}


def kda_seam(q, k, v, beta, gate, tok_start, tok_len, w, S_in, entry_head_pairs=None):
    """Seam rescan (Sec. 4.3) for the KDA row: the first ``min(w, tok_len[e])``
    tokens of entry e run through the recurrence from S_in[e].  Returns
    (o_seam [n, w, h_v, d_v] with rows past w_eff NaN, S_post [n, h_v, d_k, d_v])."""
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
        o_eh, S_eh = kda_recurrence(q[lo:hi, g], k[lo:hi, g], v[lo:hi, h], beta[lo:hi, h],
                                    gate[lo:hi, h], S0=S_in[e, h])
        o_seam[e, :hi - lo, h] = o_eh
        S_post[e, h] = S_eh
    return o_seam, S_post
