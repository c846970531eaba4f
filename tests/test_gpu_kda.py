"""Parity of the KDA row of Tab. 1 (delta rule with a per-channel gate; Tab. 3
dense operator) through the C ABI against the float64 oracle.

Same bar as the GDN path: relative Frobenius error per (segment, head) tensor,
1e-4 for float32 inputs and 1e-2 for bf16 inputs with float32 accumulation.
Tab. 3 fixes the operator T_C, not how a cache splits it into a scalar and a
matrix, so the operator is compared as T_C: exp(ld_gpu - ld_ref) P_hat_gpu
against the oracle's P_hat (in float64, so no underflow), and log_decay only as
finite and within the per-token gate extremes summed over the segment.  The tuples compose with the GDN composition
(hypic_compose_segments).  Every test prints its case before touching the GPU.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import gdn as G
from oracle import kda as K
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


def _workload(lengths, heads, d, dt, kind="softplus", seed=21):
    w = W.segment_workload(2, lengths=lengths, heads=heads, d=d, dtype=dt, seed=seed)
    T = int(w["cu_seqlens"][-1])
    w["gate"] = W.family_gate("diagonal", T, heads[1], d, seed + 1000, kind=kind)
    return w


def _dev(w, dt):
    tdt = torch.bfloat16 if dt == W.BF16 else torch.float32
    q, k, v = [torch.from_numpy(w[key]).cuda().to(tdt).contiguous() for key in ("q", "k", "v")]
    beta = torch.from_numpy(w["beta"]).cuda().contiguous()
    gate = torch.from_numpy(w["gate"]).cuda().contiguous()
    return q, k, v, beta, gate


def tc_error(P_gpu, ld_gpu, P_ref, ld_ref):
    """Relative Frobenius error of T_C = exp(log_decay) P_hat between two
    splits, formed as exp(ld_gpu - ld_ref) P_gpu against P_ref."""
    return rel(np.exp(float(ld_gpu) - float(ld_ref)) * P_gpu, P_ref)


def check_log_decay(ld, gate):
    """A cache's scalar split is free (Tab. 3 fixes T_C only); the kernel's
    must be finite and lie between the per-token smallest and largest gates
    summed over the segment."""
    lo = float(np.sum(np.min(gate, axis=1))) if len(gate) else 0.0
    hi = float(np.sum(np.max(gate, axis=1))) if len(gate) else 0.0
    slack = 1e-4 * (1.0 + abs(lo))
    return np.isfinite(ld) and lo - slack <= ld <= hi + slack


def _check_build(res, ref, cu, pairs, tol, tag, gate, operator=True):
    o, S = _np(res["o"]), _np(res["S_seg"])
    worst = {"o": 0.0, "S": 0.0}
    if operator:
        worst.update({"T_C": 0.0})
        P, ld = _np(res["P_hat"]), _np(res["log_decay"])
    for s, h in pairs:
        lo, hi = int(cu[s]), int(cu[s + 1])
        if hi > lo:
            worst["o"] = max(worst["o"], rel(o[lo:hi, h], ref["o"][lo:hi, h]))
        worst["S"] = max(worst["S"], rel(S[s, h], ref["S_seg"][s, h]))
        if operator:
            worst["T_C"] = max(worst["T_C"], tc_error(P[s, h], ld[s, h], ref["P_hat"][s, h],
                                                      ref["log_decay"][s, h]))
            assert check_log_decay(ld[s, h], gate[lo:hi, h]), (tag, s, h, ld[s, h])
    print("%s max err: %s" % (tag, {k: "%.2e" % v for k, v in worst.items()}), flush=True)
    for key, val in worst.items():
        assert val <= tol, (tag, key, val)


CASES = [
    # dtype, d_k = d_v, heads (qk, v), gate kind
    (W.F32, 64, (1, 2), "softplus"),
    (W.F32, 128, (2, 2), "logsigmoid"),
    (W.BF16, 128, (2, 4), "softplus"),
    (W.BF16, 64, (2, 2), "logsigmoid"),
]


@pytest.mark.parametrize("dt,d,heads,kind", CASES)
def test_kda_build_compose_seam(hy, dt, d, heads, kind):
    lengths = [150, 64, 0, 1, 97, 200]
    _say("kda %s d=%d heads=%s gate=%s lengths=%s: build + compose + seam"
         % (dt, d, heads, kind, lengths))
    w = _workload(lengths, heads, d, dt, kind)
    cu = w["cu_seqlens"]
    q, k, v, beta, gate = _dev(w, dt)
    res = hy.kda_build(q, k, v, beta, gate, cu)
    n_seg, h_v = len(lengths), heads[1]
    # two requests: segments 4, 0, 5, 1 behind a prefix, and 3, 2 from zero
    ids = np.array([4, 0, 5, 1, 3, 2], dtype=np.int32)
    offs = np.array([0, 4, 6], dtype=np.int32)
    rng = np.random.default_rng(5)
    prefix = (rng.standard_normal((2, h_v, d, d)) * 0.3).astype(np.float32)
    prefix[1] = 0.0
    S_out, S_inc = hy.compose_segments(res["P_hat"], res["log_decay"], res["S_seg"], ids, offs,
                                       S_prefix=torch.from_numpy(prefix).cuda())
    lens = np.diff(cu)
    keep = lens[ids] > 0
    sid = ids[keep]
    inc = S_inc[torch.as_tensor(np.nonzero(keep)[0], device="cuda")].contiguous()
    seams = {sw: hy.kda_seam(q, k, v, beta, gate, cu[:-1][sid], lens[sid], sw, inc)
             for sw in (8, 100)}
    torch.cuda.synchronize()

    tol = TOL[dt]
    ref = K.kda_build_segments(w["q"], w["k"], w["v"], w["beta"], w["gate"], cu)
    pairs = [(s, h) for s in range(n_seg) for h in range(h_v)]
    _check_build(res, ref, cu, pairs, tol, "kda %s build" % dt, w["gate"])
    R_out, R_inc = G.compose(ref["P_hat"], ref["log_decay"], ref["S_seg"], ids, offs,
                             S_prefix=prefix)
    for r in range(2):
        for h in range(h_v):
            assert rel(_np(S_out)[r, h], R_out[r, h]) <= tol, (r, h)
    for j in range(len(ids)):
        for h in range(h_v):
            assert rel(_np(S_inc)[j, h], R_inc[j, h]) <= tol, (j, h)
    R_keep = R_inc[np.nonzero(keep)[0]]
    for sw, (o_seam, S_post) in seams.items():
        R_o, R_post = K.kda_seam(w["q"], w["k"], w["v"], w["beta"], w["gate"], cu[:-1][sid],
                                 lens[sid], sw, R_keep)
        og, Sp = _np(o_seam), _np(S_post)
        for e in range(len(sid)):
            we = min(sw, int(lens[sid[e]]))
            for h in range(h_v):
                assert rel(og[e, :we, h], R_o[e, :we, h]) <= tol, (sw, e, h)
                assert rel(Sp[e, h], R_post[e, h]) <= tol, (sw, e, h)


def test_kda_more_segments_than_the_inline_order(hy):
    """150 segments: past 128 the longest-first order of both launches is
    ranked on the device into the workspace; every (segment, head) lands on
    its own rows, operator included."""
    rng = np.random.default_rng(38)
    lengths = [int(x) for x in rng.integers(0, 131, size=150)]
    lengths[3] = 0
    lengths[120] = 130
    _say("kda bf16 d=128 heads=(1, 2), %d segments (%d tokens)" % (len(lengths), sum(lengths)))
    w = W.segment_workload(2, lengths=lengths, heads=(1, 2), d=128, dtype=W.BF16, seed=39)
    T = int(w["cu_seqlens"][-1])
    w["gate"] = W.family_gate("diagonal", T, 2, 128, 1039)
    q, k, v, beta, gate = _dev(w, W.BF16)
    res = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"])
    torch.cuda.synchronize()
    ref = K.kda_build_segments(w["q"], w["k"], w["v"], w["beta"], w["gate"], w["cu_seqlens"])
    pairs = [(s, h) for s in range(len(lengths)) for h in range(2)]
    _check_build(res, ref, w["cu_seqlens"], pairs, TOL[W.BF16], "kda 150 segments", w["gate"])


def test_kda_without_operator_matches_with(hy):
    """P_hat = NULL skips the operator columns; o and S_seg are unchanged."""
    _say("kda bf16 d=128 build without the operator")
    w = _workload([130, 70], (2, 2), 128, W.BF16)
    q, k, v, beta, gate = _dev(w, W.BF16)
    a = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"])
    b = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"], want_operator=False)
    torch.cuda.synchronize()
    assert b["P_hat"] is None
    assert torch.equal(a["o"], b["o"]) and torch.equal(a["S_seg"], b["S_seg"])


def test_kda_composed_state_equals_concatenation(hy):
    """Eq. (6) on the GPU: the composed tuples of consecutive segments equal the
    oracle's recurrence over the whole concatenation (float32)."""
    lengths = [128, 70, 200]
    _say("kda f32 d=64 composed state vs concatenation %s" % lengths)
    w = _workload(lengths, (1, 1), 64, W.F32)
    q, k, v, beta, gate = _dev(w, W.F32)
    res = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"])
    S_out, _ = hy.compose_segments(res["P_hat"], res["log_decay"], res["S_seg"], [0, 1, 2],
                                   [0, 3])
    torch.cuda.synchronize()
    _, S_full = K.kda_recurrence(w["q"][:, 0], w["k"][:, 0], w["v"][:, 0], w["beta"][:, 0],
                                 w["gate"][:, 0])
    assert rel(_np(S_out)[0, 0], S_full) <= TOL[W.F32]


@pytest.mark.parametrize("dt", [W.F32, W.BF16])
def test_kda_with_channel_uniform_gates_matches_the_gdn_build(hy, dt):
    """With the same gate on every channel the KDA row is the GDN row: the KDA
    build equals the GDN build of the same tokens (o, S_seg, and T_C through
    both factorisations)."""
    _say("kda vs gdn build, channel-uniform gates, %s d=128" % dt)
    w = W.segment_workload(2, lengths=[150, 64, 97], heads=(2, 4), d=128, dtype=dt, seed=31)
    T, h_v = int(w["cu_seqlens"][-1]), 4
    w["gate"] = np.repeat(w["log_alpha"][:, :, None], 128, axis=2).astype(np.float32)
    q, k, v, beta, gate = _dev(w, dt)
    la = torch.from_numpy(w["log_alpha"]).cuda().contiguous()
    a = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"])
    b = hy.build_segment(q, k, v, beta, la, w["cu_seqlens"])
    torch.cuda.synchronize()
    tol = TOL[dt]
    assert rel(_np(a["o"]), _np(b["o"])) <= tol
    for s in range(3):
        for h in range(h_v):
            assert rel(_np(a["S_seg"])[s, h], _np(b["S_seg"])[s, h]) <= tol
            Ta = np.exp(_np(a["log_decay"])[s, h]) * _np(a["P_hat"])[s, h]
            Tb = np.exp(_np(b["log_decay"])[s, h]) * _np(b["P_hat"])[s, h]
            assert rel(Ta, Tb) <= tol, (s, h)


def test_kda_fullsize_layer_sampled(hy):
    """16 heads, d = 128, 8 x 2048 bf16 tokens: sampled (segment, head) pairs
    against the oracle; one full request composed from the GPU's own tuples."""
    _say("kda layer-bf16 16 heads d=128 8x2048: sampled pairs")
    w = W.segment_workload(2)
    T = int(w["cu_seqlens"][-1])
    w["gate"] = W.family_gate("diagonal", T, 16, 128, w["seed"] + 2000)
    cu = w["cu_seqlens"]
    q, k, v, beta, gate = _dev(w, W.BF16)
    res = hy.kda_build(q, k, v, beta, gate, cu)
    ids = np.arange(8, dtype=np.int32)
    S_out, _ = hy.compose_segments(res["P_hat"], res["log_decay"], res["S_seg"], ids, [0, 8])
    torch.cuda.synchronize()
    pairs = [(0, 0), (3, 7), (7, 15)]
    ref = K.kda_build_segments(w["q"], w["k"], w["v"], w["beta"], w["gate"], cu,
                               seg_head_pairs=pairs)
    _check_build(res, ref, cu, pairs, TOL[W.BF16], "kda layer", w["gate"])
    R_out, _ = G.compose(_np(res["P_hat"]), _np(res["log_decay"]), _np(res["S_seg"]), ids,
                         [0, 8], req_head_pairs=[(0, 9)])
    assert rel(_np(S_out)[0, 9], R_out[0, 9]) <= 1e-5


def test_kda_build_is_deterministic(hy):
    _say("kda bf16 determinism")
    w = _workload([300, 40, 129], (2, 4), 128, W.BF16)
    q, k, v, beta, gate = _dev(w, W.BF16)
    a = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"])
    b = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"])
    torch.cuda.synchronize()
    for key in ("o", "S_seg", "P_hat", "log_decay"):
        assert torch.equal(a[key], b[key]), key


def test_kda_prebound_pipeline_equals_ops(hy):
    """The pre-bound build the bench times gives exactly the tuple of kda_build."""
    _say("kda bf16 pre-bound pipeline against kda_build")
    from paper_2607_01299_amd.pipeline import KdaPipeline
    w = _workload([300, 40, 129], (2, 4), 128, W.BF16)
    q, k, v, beta, gate = _dev(w, W.BF16)
    a = hy.kda_build(q, k, v, beta, gate, w["cu_seqlens"])
    pipe = KdaPipeline(q, k, v, beta, gate, w["cu_seqlens"])
    pipe.build()
    torch.cuda.synchronize()
    for key in ("o", "S_seg", "P_hat", "log_decay"):
        assert torch.equal(a[key], getattr(pipe, key)), key
