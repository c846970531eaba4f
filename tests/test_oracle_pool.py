"""The spawned-worker oracle pool that the full-size parity tests use returns
exactly what a direct oracle call returns."""

import numpy as np

import oracle
from _oracle_pool import build_pairs


def test_pool_matches_direct_oracle_calls():
    rng = np.random.default_rng(0)
    probs = []
    for L in (5, 70, 130):
        q = rng.standard_normal((L, 1, 16))
        k = rng.standard_normal((L, 1, 16))
        q /= np.linalg.norm(q, axis=-1, keepdims=True)
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
        v = rng.standard_normal((L, 1, 16))
        b = rng.uniform(0, 1, (L, 1))
        a = np.log(rng.uniform(0.9, 1, (L, 1)))
        probs.append((q, k, v, b, a))
    for p, (o, S, P, ld) in zip(probs, build_pairs(probs)):
        ref = oracle.build_segments(*p, [0, p[0].shape[0]])
        assert np.array_equal(o, ref["o"][:, 0])
        assert np.array_equal(S, ref["S_seg"][0, 0])
        assert np.array_equal(P, ref["P_hat"][0, 0])
        assert ld == ref["log_decay"][0, 0]
