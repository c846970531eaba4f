"""Parity of the scalar and diagonal transition families (Tab. 1 rows, Tab. 3
compressed operators) through the C ABI against the float64 oracle.

Same bar as the GDN path: relative Frobenius error per (segment, head) tensor,
1e-4 for float32 inputs and 1e-2 for bf16 inputs with float32 accumulation;
log_decay by its absolute error.  Every test prints its case before touching
the GPU.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import families as F
from paper_2607_01299_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = {W.F32: 1e-4, W.BF16: 1e-2}


def _say(msg):
    print("[case] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def hy():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2607_01299_amd as hy
    from paper_2607_01299_amd import _lib
    _lib.load()
    return hy


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel(x, ref):
    nr = np.linalg.norm(ref)
    if nr == 0.0:
        return float(np.linalg.norm(x))
    return float(np.linalg.norm(x - ref) / nr)


def _tok(w, dt):
    tdt = torch.bfloat16 if dt == W.BF16 else torch.float32
    return [torch.from_numpy(w[key]).cuda().to(tdt).contiguous() for key in ("q", "k", "v")]


def _workload(family, lengths, heads, d, dt, kind="softplus", seed=11):
    w = W.segment_workload(2, lengths=lengths, heads=heads, d=d, dtype=dt, seed=seed)
    T = int(w["cu_seqlens"][-1])
    w["gate"] = W.family_gate(family, T, heads[1], d, seed + 1000, kind=kind)
    return w


def _check_build(res, ref, cu, pairs, tol, tag):
    o, S, ld = _np(res["o"]), _np(res["S_seg"]), _np(res["log_decay"])
    worst = {"o": 0.0, "S": 0.0, "ld": 0.0}
    for s, h in pairs:
        lo, hi = int(cu[s]), int(cu[s + 1])
        if hi > lo:
            worst["o"] = max(worst["o"], rel(o[lo:hi, h], ref["o"][lo:hi, h]))
        worst["S"] = max(worst["S"], rel(S[s, h], ref["S_seg"][s, h]))
        worst["ld"] = max(worst["ld"], float(np.max(np.abs(ld[s, h] - ref["log_decay"][s, h]))))
    print("%s max err: %s" % (tag, {k: "%.2e" % v for k, v in worst.items()}), flush=True)
    for key, val in worst.items():
        assert val <= tol, (tag, key, val)


CASES = [
    # family, dtype, d_k = d_v, heads (qk, v), gate kind
    ("scalar", W.F32, 64, (1, 2), "softplus"),
    ("scalar", W.BF16, 128, (2, 4), "softplus"),
    ("scalar", W.BF16, 128, (4, 4), "retnet"),
    ("diagonal", W.F32, 64, (1, 2), "softplus"),
    ("diagonal", W.BF16, 128, (2, 4), "softplus"),
    ("diagonal", W.BF16, 64, (2, 2), "logsigmoid"),
    ("diagonal", W.BF16, 128, (2, 2), "logsigmoid"),
    ("diagonal", W.F32, 128, (2, 2), "logsigmoid"),
]


@pytest.mark.parametrize("family,dt,d,heads,kind", CASES)
def test_family_build_compose_seam(hy, family, dt, d, heads, kind):
    lengths = [150, 64, 0, 1, 97, 200]
    _say("family %s %s d=%d heads=%s gate=%s lengths=%s: build + compose + seam"
         % (family, dt, d, heads, kind, lengths))
    w = _workload(family, lengths, heads, d, dt, kind)
    cu = w["cu_seqlens"]
    q, k, v = _tok(w, dt)
    gate = torch.from_numpy(w["gate"]).cuda().contiguous()
    res = hy.family_build(family, q, k, v, gate, cu)
    n_seg, h_v = len(lengths), heads[1]
    # two requests: segments 4, 0, 5, 1 behind a prefix, and 3, 2 from zero
    ids = np.array([4, 0, 5, 1, 3, 2], dtype=np.int32)
    offs = np.array([0, 4, 6], dtype=np.int32)
    rng = np.random.default_rng(5)
    prefix = (rng.standard_normal((2, h_v, d, d)) * 0.3).astype(np.float32)
    prefix[1] = 0.0
    S_out, S_inc = hy.family_compose(family, res["log_decay"], res["S_seg"], ids, offs,
                                     S_prefix=torch.from_numpy(prefix).cuda())
    lens = np.diff(cu)
    seam = {}
    for sw in (8, 100):
        keep = lens[ids] > 0
        seam[sw] = (ids[keep], hy.family_seam(family, q, k, v, gate, cu[:-1][ids[keep]],
                                              lens[ids[keep]], sw,
                                              S_inc[torch.as_tensor(np.nonzero(keep)[0],
                                                                    device="cuda")].contiguous()))
    torch.cuda.synchronize()

    tol = TOL[dt]
    ref = F.family_build_segments(family, w["q"], w["k"], w["v"], w["gate"], cu)
    pairs = [(s, h) for s in range(n_seg) for h in range(h_v)]
    _check_build(res, ref, cu, pairs, tol, "%s %s build" % (family, dt))
    R_out, R_inc = F.family_compose(family, ref["log_decay"], ref["S_seg"], ids, offs,
                                    S_prefix=prefix)
    for r in range(2):
        for h in range(h_v):
            assert rel(_np(S_out)[r, h], R_out[r, h]) <= tol
    for j in range(len(ids)):
        for h in range(h_v):
            assert rel(_np(S_inc)[j, h], R_inc[j, h]) <= tol, (j, h)
    for sw, (sid, (o_seam, S_post)) in seam.items():
        keep = np.nonzero(lens[ids] > 0)[0]
        R_o, R_post = F.family_seam(family, w["q"], w["k"], w["v"], w["gate"], cu[:-1][sid],
                                    lens[sid], sw, R_inc[keep])
        og, Sp = _np(o_seam), _np(S_post)
        for e in range(len(sid)):
            we = min(sw, int(lens[sid[e]]))
            for h in range(h_v):
                assert rel(og[e, :we, h], R_o[e, :we, h]) <= tol, (sw, e, h)
                assert rel(Sp[e, h], R_post[e, h]) <= tol, (sw, e, h)


@pytest.mark.parametrize("family", ["scalar", "diagonal"])
def test_family_composed_state_equals_concatenation(hy, family):
    """Eq. (6) on the GPU: composing the built tuples of consecutive segments
    equals the oracle's recurrence over the whole concatenation (float32)."""
    lengths = [128, 70, 200]
    _say("family %s f32 d=64 composed state vs concatenation %s" % (family, lengths))
    w = _workload(family, lengths, (1, 1), 64, W.F32)
    cu = w["cu_seqlens"]
    q, k, v = _tok(w, W.F32)
    gate = torch.from_numpy(w["gate"]).cuda().contiguous()
    res = hy.family_build(family, q, k, v, gate, cu)
    S_out, _ = hy.family_compose(family, res["log_decay"], res["S_seg"], [0, 1, 2], [0, 3])
    torch.cuda.synchronize()
    g = w["gate"][:, 0]
    _, S_full = F.family_recurrence(family, w["q"][:, 0], w["k"][:, 0], w["v"][:, 0], g)
    assert rel(_np(S_out)[0, 0], S_full) <= TOL[W.F32]


@pytest.mark.parametrize("family", ["scalar", "diagonal"])
def test_family_fullsize_layer_sampled(hy, family):
    """16 heads, d = 128, 8 x 2048 bf16 tokens: sampled (segment, head) pairs
    against the oracle, one full request composed."""
    _say("family %s layer-bf16 16 heads d=128 8x2048: sampled pairs" % family)
    w = W.segment_workload(2)
    T = int(w["cu_seqlens"][-1])
    w["gate"] = W.family_gate(family, T, 16, 128, w["seed"] + 1000)
    cu = w["cu_seqlens"]
    q, k, v = _tok(w, W.BF16)
    gate = torch.from_numpy(w["gate"]).cuda().contiguous()
    res = hy.family_build(family, q, k, v, gate, cu)
    ids = np.arange(8, dtype=np.int32)
    S_out, S_inc = hy.family_compose(family, res["log_decay"], res["S_seg"], ids, [0, 8])
    torch.cuda.synchronize()
    pairs = [(0, 0), (3, 7), (7, 15), (5, 9)]
    ref = F.family_build_segments(family, w["q"], w["k"], w["v"], w["gate"], cu,
                                  seg_head_pairs=pairs)
    _check_build(res, ref, cu, pairs, TOL[W.BF16], "%s layer" % family)
    # composition of the GPU's own tuples, head 9, against the oracle's compose
    ld = _np(res["log_decay"])
    S = _np(res["S_seg"])
    R_out, _ = F.family_compose(family, ld, S, ids, [0, 8], req_head_pairs=[(0, 9)])
    assert rel(_np(S_out)[0, 9], R_out[0, 9]) <= 1e-5


def test_family_build_is_deterministic(hy):
    _say("family diagonal bf16 determinism")
    w = _workload("diagonal", [300, 40, 129], (2, 4), 128, W.BF16)
    q, k, v = _tok(w, W.BF16)
    gate = torch.from_numpy(w["gate"]).cuda().contiguous()
    a = hy.family_build("diagonal", q, k, v, gate, w["cu_seqlens"])
    b = hy.family_build("diagonal", q, k, v, gate, w["cu_seqlens"])
    torch.cuda.synchronize()
    for key in ("o", "S_seg", "log_decay"):
        assert torch.equal(a[key], b[key]), key
