"""Float64 oracle: token-by-token gated delta rule, segment operator, Eq. (6)
composition and seam rescan.

TEST INFRASTRUCTURE ONLY (see the package docstring): this module defines what
the HIP path must reproduce and is never used by it.

Notation follows the paper (Hypic, arXiv 2607.01299):

* per head the state is ``S`` in R^{d_k x d_v};
* per token t: ``q_t, k_t`` in R^{d_k}, ``v_t`` in R^{d_v}, scalars ``beta_t`` and
  ``a_t = log(alpha_t)`` (the gate ``g_t`` of Tab. 1 is ``alpha_t = exp(a_t)``);
* the GDN row of Tab. 1 gives the transition ``T_t = alpha_t (I - beta_t k_t k_t^T)``
  and the write ``u_t = beta_t k_t v_t^T`` of the unified recurrence Eq. (2):
  ``S_t = T_t S_{t-1} + u_t`` and ``o_t = S_t^T q_t`` (the token reads the state
  after its own write; no scale factor is applied).

Readings of points the paper leaves open:

* the segment operator ``T_C`` multiplies later tokens on the left, as in Eq. (4)
  and the product convention stated under Eq. (6);
* ``T_C`` is kept factored the way Tab. 3 writes the GDN closed form,
  ``T_C = exp(log_decay) * P_hat`` with ``log_decay = sum_t a_t`` and
  ``P_hat = prod_t (I - beta_t k_t k_t^T)``;
* grouped heads: v-head ``h`` reads qk-head ``h // (h_v // h_qk)``.

All arithmetic is numpy float64.  Inputs may be float32 (or bf16 values held in
float32); they are upcast exactly.
"""

import numpy as np


def qk_head_of(h, h_v, h_qk):
    """qk-head read by v-head ``h`` when ``h_v`` value heads share ``h_qk`` key
    heads in contiguous groups (the paper is silent on grouping)."""
    if h_v % h_qk != 0:
        raise ValueError("h_v must be a multiple of h_qk")
    return h // (h_v // h_qk)


def recurrence(q, k, v, beta, log_alpha, S0=None):
    """Run the GDN recurrence of Eq. (2) (Tab. 1, GDN row) over one head.

    q, k: [L, d_k]; v: [L, d_v]; beta, log_alpha: [L]; S0: [d_k, d_v] or None
    (zero start).  For each token, in order:

        S <- alpha_t (I - beta_t k_t k_t^T) S + beta_t k_t v_t^T
        o_t = S^T q_t

    Returns (o [L, d_v], S_end [d_k, d_v]) in float64.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    log_alpha = np.asarray(log_alpha, dtype=np.float64)
    L, d_k = k.shape
    d_v = v.shape[1]
    S = np.zeros((d_k, d_v)) if S0 is None else np.array(S0, dtype=np.float64)
    o = np.zeros((L, d_v))
    for t in range(L):
        kt = k[t]
        # T_t S = alpha_t (S - beta_t k_t (k_t^T S))
        S = np.exp(log_alpha[t]) * (S - beta[t] * np.outer(kt, kt @ S))
        # + u_t
        S = S + beta[t] * np.outer(kt, v[t])
        o[t] = S.T @ q[t]
    return o, S


def segment_operator(k, beta, log_alpha):
    """Segment-cumulative transition operator of one head, factored.

    The paper obtains ``T_C`` by running the same recurrence a second time with
    the initial state set to the identity and every write zeroed, since the
    product of the per-token transitions applied to I is T_C (Sec. 5, state
    construction).  The same is done here for the decay-free factor
    ``P_hat = prod_t (I - beta_t k_t k_t^T)`` (gate set to 1), and the scalar gate
    product of the Tab. 3 GDN closed form is carried as ``log_decay = sum_t a_t``,
    so that ``T_C = exp(log_decay) * P_hat``.

    Returns (P_hat [d_k, d_k], log_decay float) in float64.
    """
    k = np.asarray(k, dtype=np.float64)
    L, d_k = k.shape
    _, P_hat = recurrence(
        q=np.zeros((L, d_k)),
        k=k,
        v=np.zeros((L, d_k)),
        beta=beta,
        log_alpha=np.zeros(L),
        S0=np.eye(d_k),
    )
    log_decay = float(np.sum(np.asarray(log_alpha, dtype=np.float64)))
    return P_hat, log_decay


def build_segments(q, k, v, beta, log_alpha, cu_seqlens, want_operator=True,
                   seg_head_pairs=None):
    """Zero-start build of every segment in a packed batch (Sec. 4.2 cache tuple).

    q, k: [T, h_qk, d_k]; v: [T, h_v, d_v]; beta, log_alpha: [T, h_v];
    cu_seqlens: [n_seg + 1] token offsets.  Segments are independent: each starts
    from S = 0 (insight 1 of Sec. 3.1, the tuple depends only on the segment's own
    tokens).

    ``seg_head_pairs`` (optional list of (segment, v-head)) restricts the work to
    those pairs; the other entries of the outputs are left as NaN.

    Returns dict with o [T, h_v, d_v], S_seg [n_seg, h_v, d_k, d_v],
    P_hat [n_seg, h_v, d_k, d_k], log_decay [n_seg, h_v] (float64).
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
        o_sh, S_sh = recurrence(q[lo:hi, g], k[lo:hi, g], v[lo:hi, h],
                                beta[lo:hi, h], log_alpha[lo:hi, h])
        o[lo:hi, h] = o_sh
        S_seg[s, h] = S_sh
        if want_operator:
            P_hat[s, h], log_decay[s, h] = segment_operator(
                k[lo:hi, g], beta[lo:hi, h], log_alpha[lo:hi, h])
    return {"o": o, "S_seg": S_seg, "P_hat": P_hat, "log_decay": log_decay}


def compose(P_hat, log_decay, S_seg, seg_ids, req_offsets, S_prefix=None,
            req_head_pairs=None):
    """Chain cached segment tuples behind a prefix state, Eq. (6).

    Request ``r`` applies segments ``seg_ids[req_offsets[r]:req_offsets[r+1]]`` in
    that order.  Eq. (6) is evaluated as repeated application of the two-segment
    true splice of Eq. (4): starting from the prefix end-state (zero when
    ``S_prefix`` is None), each listed segment i maps the running state S to
    ``T_{C_i} S + S_{C_i|0}`` with ``T_{C_i} = exp(log_decay_i) * P_hat_i``.

    Returns (S_out [n_req, h_v, d_k, d_v], S_incoming [nnz, h_v, d_k, d_v]) where
    ``S_incoming[j]`` is the running state just before listed segment j is applied.
    ``req_head_pairs`` optionally restricts the work (others stay NaN).
    """
    P_hat = np.asarray(P_hat)
    S_seg = np.asarray(S_seg)
    log_decay = np.asarray(log_decay, dtype=np.float64)
    n_pool, h_v, d_k, d_v = S_seg.shape
    offs = [int(x) for x in req_offsets]
    ids = [int(x) for x in seg_ids]
    n_req = len(offs) - 1
    S_out = np.full((n_req, h_v, d_k, d_v), np.nan)
    S_inc = np.full((len(ids), h_v, d_k, d_v), np.nan)
    if req_head_pairs is None:
        req_head_pairs = [(r, h) for r in range(n_req) for h in range(h_v)]
    for r, h in req_head_pairs:
        if S_prefix is None:
            S = np.zeros((d_k, d_v))
        else:
            S = np.array(S_prefix[r, h], dtype=np.float64)
        for j in range(offs[r], offs[r + 1]):
            i = ids[j]
            S_inc[j, h] = S
            T_i = np.exp(log_decay[i, h]) * np.asarray(P_hat[i, h], dtype=np.float64)
            S = T_i @ S + np.asarray(S_seg[i, h], dtype=np.float64)
        S_out[r, h] = S
    return S_out, S_inc


def seam(q, k, v, beta, log_alpha, tok_start, tok_len, w, S_in,
         entry_head_pairs=None):
    """Seam-window rescan through a linear-attention layer (Sec. 4.3, seam
    propagation): the first ``w_eff = min(w, tok_len[e])`` tokens of entry ``e``
    are run through the recurrence of Eq. (2) starting from the composed state
    ``S_in[e]``, emitting their per-token outputs and the advanced state.

    q, k: [T, h_qk, d_k]; v: [T, h_v, d_v]; beta, log_alpha: [T, h_v];
    S_in: [n_entries, h_v, d_k, d_v].
    Returns (o_seam [n_entries, w, h_v, d_v] with rows >= w_eff NaN,
    S_post [n_entries, h_v, d_k, d_v]).
    """
    T, h_qk, d_k = np.shape(k)
    h_v, d_v = np.shape(v)[1], np.shape(v)[2]
    n_e = len(tok_start)
    o_seam = np.full((n_e, w, h_v, d_v), np.nan)
    S_post = np.full((n_e, h_v, d_k, d_v), np.nan)
    if entry_head_pairs is None:
        entry_head_pairs = [(e, h) for e in range(n_e) for h in range(h_v)]
    for e, h in entry_head_pairs:
        lo = int(tok_start[e])
        w_eff = min(int(w), int(tok_len[e]))
        g = qk_head_of(h, h_v, h_qk)
        o_eh, S_eh = recurrence(q[lo:lo + w_eff, g], k[lo:lo + w_eff, g],
                                v[lo:lo + w_eff, h], beta[lo:lo + w_eff, h],
                                log_alpha[lo:lo + w_eff, h], S0=S_in[e, h])
        o_seam[e, :w_eff, h] = o_eh
        S_post[e, h] = S_eh
    return o_seam, S_post


def compose_with_seams(P_tail, log_decay_tail, S_tail, q, k, v, beta, log_alpha, seam_start,
                       seam_len, w, seg_ids, req_offsets, S_prefix=None, req_head_pairs=None):
    """Reuse with seam windows that advance the state (Sec. 4.3: the seam is left
    out of the cached tuple and, at reuse, recomputed through the layer from the
    composed state).

    Pool entry ``i`` is cached as the tuple of its tail, tokens
    ``[seam_start[i] + w_i, seam_start[i] + seam_len[i])`` with
    ``w_i = min(w, seam_len[i])`` (``P_tail, log_decay_tail, S_tail`` are built over
    those tokens), and its seam is its first ``w_i`` tokens.  For request ``r``,
    starting from the prefix state (zero when None), each listed entry ``i`` in
    order runs its seam tokens through the recurrence of Eq. (2) from the
    running state (emitting their outputs and advancing the state), then applies
    its tail tuple by Eq. (4): ``S <- exp(log_decay_i) P_tail_i S + S_tail_i``.

    Returns (S_out [n_req, h_v, d_k, d_v], o_seam [nnz, w, h_v, d_v] (rows past
    w_i NaN), S_incoming [nnz, h_v, d_k, d_v], the state entering each listed
    entry's seam), in the CSR order of ``seg_ids``.
    """
    T, h_qk, d_k = np.shape(k)
    h_v, d_v = np.shape(v)[1], np.shape(v)[2]
    offs = [int(x) for x in req_offsets]
    ids = [int(x) for x in seg_ids]
    n_req = len(offs) - 1
    S_out = np.full((n_req, h_v, d_k, d_v), np.nan)
    o_seam = np.full((len(ids), w, h_v, d_v), np.nan)
    S_inc = np.full((len(ids), h_v, d_k, d_v), np.nan)
    if req_head_pairs is None:
        req_head_pairs = [(r, h) for r in range(n_req) for h in range(h_v)]
    for r, h in req_head_pairs:
        g = qk_head_of(h, h_v, h_qk)
        S = np.zeros((d_k, d_v)) if S_prefix is None else np.array(S_prefix[r, h],
                                                                    dtype=np.float64)
        for j in range(offs[r], offs[r + 1]):
            i = ids[j]
            lo = int(seam_start[i])
            wi = min(int(w), int(seam_len[i]))
            S_inc[j, h] = S
            o_seam[j, :wi, h], S = recurrence(q[lo:lo + wi, g], k[lo:lo + wi, g],
                                              v[lo:lo + wi, h], beta[lo:lo + wi, h],
                                              log_alpha[lo:lo + wi, h], S0=S)
            T_i = np.exp(log_decay_tail[i, h]) * np.asarray(P_tail[i, h], dtype=np.float64)
            S = T_i @ S + np.asarray(S_tail[i, h], dtype=np.float64)
        S_out[r, h] = S
    return S_out, o_seam, S_inc
