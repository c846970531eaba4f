"""Degenerate inputs of the gated delta rule through the segment build
(hypic_build_segment), checked against closed forms the recurrence fixes
(Sec. 4.1, Eq. (4)) and against the float64 oracle:

* beta = 0: no token writes, so every transition is alpha_t I: P_hat is the
  identity and S_seg and o are zero, bit for bit; log_decay is sum log alpha;
* alpha = 1 (log_alpha = 0): no decay, log_decay is exactly 0;
* one key for every token (alpha = 1): the product of (I - beta_t k k^T) is
  I - ((1 - prod_t (1 - beta_t |k|^2)) / |k|^2) k k^T;
* q = 0: every output is zero, the states are the oracle's;
* a 16384-token segment with slow decay and one without decay: the
  normalised operator (a product of 16384 contractions, Frobenius norm near
  1e-18) and the state stay within the bound over 256 chunks.
"""

import numpy as np
import pytest
import torch

import oracle

from test_gpu_parity import _np, _say, rel

pytestmark = pytest.mark.gpu

TOL = {torch.float32: 1e-4, torch.bfloat16: 1e-2}


@pytest.fixture(scope="module")
def hy():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2607_01299_amd as hy
    from paper_2607_01299_amd import _lib
    _lib.load()
    return hy


def _tokens(rng, T, d, dt, beta=None, log_alpha=None, same_key=False, q_zero=False):
    """One head of T tokens: unit q and k, N(0,1) v, in dt (rounded once), and
    the float64 values the oracle sees."""
    q = rng.standard_normal((T, 1, d))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    if q_zero:
        q[:] = 0.0
    if same_key:
        k0 = rng.standard_normal(d)
        k = np.broadcast_to(k0 / np.linalg.norm(k0), (T, 1, d)).copy()
    else:
        k = rng.standard_normal((T, 1, d))
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, 1, d))
    b = rng.uniform(0.05, 0.95, (T, 1)) if beta is None else np.full((T, 1), beta)
    a = (np.log(rng.uniform(0.9, 1.0, (T, 1))) if log_alpha is None
         else np.full((T, 1), log_alpha))
    dev = {}
    host = {}
    for name, x in (("q", q), ("k", k), ("v", v)):
        t = torch.from_numpy(x.astype(np.float32)).to(dt).cuda().contiguous()
        dev[name] = t
        host[name] = t.float().cpu().numpy().astype(np.float64)
    for name, x in (("beta", b), ("log_alpha", a)):
        t = torch.from_numpy(x.astype(np.float32)).cuda().contiguous()
        dev[name] = t
        host[name] = t.cpu().numpy().astype(np.float64)
    return dev, host


def _build(hy, dev, T):
    res = hy.build_segment(dev["q"], dev["k"], dev["v"], dev["beta"], dev["log_alpha"],
                           np.array([0, T], dtype=np.int32))
    torch.cuda.synchronize()
    return res


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32])
def test_zero_beta_is_pure_decay(hy, dt):
    _say("degenerate: beta = 0, %s, 300 tokens" % dt)
    rng = np.random.default_rng(11)
    T, d = 300, 128
    dev, host = _tokens(rng, T, d, dt, beta=0.0)
    res = _build(hy, dev, T)
    assert torch.equal(res["P_hat"][0, 0], torch.eye(d, device="cuda"))
    assert torch.count_nonzero(res["S_seg"]).item() == 0
    assert torch.count_nonzero(res["o"].float()).item() == 0
    ld = float(res["log_decay"][0, 0])
    want = float(np.sum(host["log_alpha"]))
    assert abs(ld - want) <= 1e-5 * abs(want), (ld, want)


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32])
def test_no_decay_has_zero_log_decay(hy, dt):
    _say("degenerate: alpha = 1, %s, 257 tokens" % dt)
    rng = np.random.default_rng(12)
    T, d = 257, 64
    dev, host = _tokens(rng, T, d, dt, log_alpha=0.0)
    res = _build(hy, dev, T)
    assert float(res["log_decay"][0, 0]) == 0.0
    ref = oracle.build_segments(host["q"], host["k"], host["v"], host["beta"],
                                host["log_alpha"], [0, T])
    tol = TOL[dt]
    assert rel(_np(res["P_hat"][0, 0]), ref["P_hat"][0, 0]) <= tol
    assert rel(_np(res["S_seg"][0, 0]), ref["S_seg"][0, 0]) <= tol
    assert rel(_np(res["o"][:, 0]), ref["o"][:, 0]) <= tol


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32])
def test_one_key_for_all_tokens(hy, dt):
    _say("degenerate: one key for 200 tokens, alpha = 1, %s" % dt)
    rng = np.random.default_rng(13)
    T, d = 200, 128
    dev, host = _tokens(rng, T, d, dt, log_alpha=0.0, same_key=True)
    res = _build(hy, dev, T)
    k0 = host["k"][0, 0]
    rho = float(k0 @ k0)
    c = (1.0 - np.prod(1.0 - host["beta"][:, 0] * rho)) / rho
    P_closed = np.eye(d) - c * np.outer(k0, k0)
    assert rel(_np(res["P_hat"][0, 0]), P_closed) <= TOL[dt]
    ref = oracle.build_segments(host["q"], host["k"], host["v"], host["beta"],
                                host["log_alpha"], [0, T])
    assert rel(_np(res["S_seg"][0, 0]), ref["S_seg"][0, 0]) <= TOL[dt]
    o = _np(res["o"][:, 0])
    if dt == torch.float32:
        assert rel(o, ref["o"][:, 0]) <= TOL[dt]
        return
    # With one key the chunk's output sums cancel: o_t = (q_t . k) s_t with
    # s_t a running average of the values, formed in the chunk from corrected
    # values nu_i = beta_i (v_i - S_{i-1}^T k) that are much larger, and from
    # q_t^T S0.  Every contribution reaches the matrix cores as bf16 operands
    # (each rounded once, 2^-9 relative), so the error of o is at most 2^-8
    # times the sum of the contributions' magnitudes, R |o| in Frobenius norm
    # (R is about 27 here, and the generic 1e-2 bound does not apply: o reads
    # 1.25e-2).  S_seg and P_hat above keep the generic bound.
    q, k, v, b = host["q"][:, 0], host["k"][:, 0], host["v"][:, 0], host["beta"][:, 0]
    S = np.zeros((d, d))
    mag = np.zeros((T, d))
    for c0 in range(0, T, 64):
        c1 = min(c0 + 64, T)
        mag[c0:c1] += np.abs(q[c0:c1]) @ np.abs(S)
        for t in range(c0, c1):
            nu = b[t] * (v[t] - S.T @ k[t])
            S = S + np.outer(k[t], nu)
            mag[t:c1] += np.abs(q[t:c1] @ k[t])[:, None] * np.abs(nu)
    R = np.linalg.norm(mag) / np.linalg.norm(ref["o"][:, 0])
    e_o = rel(o, ref["o"][:, 0])
    print("  o: rel %.2e, cancellation ratio R %.1f, bound 2^-8 R = %.2e" %
          (e_o, R, 2.0 ** -8 * R), flush=True)
    assert e_o <= 2.0 ** -8 * R


def test_zero_queries_give_zero_outputs(hy):
    _say("degenerate: q = 0, bf16, 130 tokens")
    rng = np.random.default_rng(14)
    T, d = 130, 128
    dev, host = _tokens(rng, T, d, torch.bfloat16, q_zero=True)
    res = _build(hy, dev, T)
    assert torch.count_nonzero(res["o"].float()).item() == 0
    ref = oracle.build_segments(host["q"], host["k"], host["v"], host["beta"],
                                host["log_alpha"], [0, T])
    assert rel(_np(res["S_seg"][0, 0]), ref["S_seg"][0, 0]) <= 1e-2
    assert rel(_np(res["P_hat"][0, 0]), ref["P_hat"][0, 0]) <= 1e-2


@pytest.mark.timeout(300)
@pytest.mark.parametrize("slow_decay", [True, False])
def test_long_segment_stays_bounded(hy, slow_decay):
    T, d = 16384, 128
    _say("degenerate: one %d-token segment, bf16, %s" %
         (T, "alpha ~ U(0.9, 1)" if slow_decay else "alpha = 1"))
    rng = np.random.default_rng(15 + int(slow_decay))
    dev, host = _tokens(rng, T, d, torch.bfloat16, log_alpha=None if slow_decay else 0.0)
    res = _build(hy, dev, T)
    P = _np(res["P_hat"][0, 0])
    assert np.all(np.isfinite(P)) and np.isfinite(float(res["log_decay"][0, 0]))
    # a product of contractions (unit keys, 0 < beta < 1): spectral norm at most 1
    assert np.linalg.norm(P, 2) <= 1.0 + 1e-3
    ref = oracle.build_segments(host["q"], host["k"], host["v"], host["beta"],
                                host["log_alpha"], [0, T])
    e_P = rel(P, ref["P_hat"][0, 0])
    e_S = rel(_np(res["S_seg"][0, 0]), ref["S_seg"][0, 0])
    e_o = rel(_np(res["o"][:, 0]), ref["o"][:, 0])
    e_ld = abs(float(res["log_decay"][0, 0]) - ref["log_decay"][0, 0])
    print("  |P_hat| %.2e; P %.2e S %.2e o %.2e log_decay %.2e" %
          (np.linalg.norm(P), e_P, e_S, e_o, e_ld), flush=True)
    assert max(e_P, e_S, e_o) <= 1e-2 and e_ld <= 1e-2
