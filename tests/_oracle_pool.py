"""Oracle references for many (segment, head) pairs at once, computed in
freshly spawned worker processes that import only numpy and the oracle (they
never open the GPU), so the full-size parity tests can sample widely.  Test
infrastructure: only tests import this module."""

import multiprocessing as mp

import numpy as np

WORKERS = 8


def _build_pair(args):
    import oracle
    q, k, v, b, a = args
    ref = oracle.build_segments(q, k, v, b, a, [0, q.shape[0]])
    return (ref["o"][:, 0], ref["S_seg"][0, 0], ref["P_hat"][0, 0],
            float(ref["log_decay"][0, 0]))


def build_pairs(problems):
    """One-head problems (q, k, v, beta, log_alpha), each one segment, through
    the oracle's build; returns (o, S_seg, P_hat, log_decay) per problem."""
    problems = [tuple(np.ascontiguousarray(x) for x in p) for p in problems]
    ctx = mp.get_context("spawn")
    with ctx.Pool(min(WORKERS, len(problems))) as pool:
        return pool.map(_build_pair, problems, chunksize=1)
