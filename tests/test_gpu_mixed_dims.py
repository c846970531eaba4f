"""Parity at unequal key and value widths (d_k, d_v) = (64, 128) and (128, 64),
which every build path supports: the GDN build (bf16 and float32 inputs), the
scalar and diagonal families and the KDA row, each against its float64 oracle
on ragged segments with grouped heads.  Bar: relative Frobenius error per
(segment, head) tensor, 1e-4 for float32 inputs, 1e-2 for bf16, at every
segment length.  The lengths include a one-token segment whose output row is
beta (q . k) v with q . k = 0.009 for two unit vectors in this draw: a score
that nearly cancels, which the per-channel-gate rows must form from hi + lo
operands.  KDA operators are compared as T_C (Tab. 3 fixes T_C, not its
scalar split).
"""

import sys

import numpy as np
import pytest
import torch

from oracle import families as F
from oracle import gdn as G
from oracle import kda as K
from paper_2607_01299_amd import workloads as W
from test_gpu_kda import check_log_decay, tc_error

pytestmark = pytest.mark.gpu

TOL = {W.F32: 1e-4, W.BF16: 1e-2}
DIMS = [(64, 128), (128, 64)]
LENGTHS = [70, 130, 1]


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


def _tokens(d_k, d_v, dt, seed):
    rng = np.random.default_rng(seed)
    T = sum(LENGTHS)
    w = W.draw_tokens(rng, T, 2, 4, d_k, d_v, dt)
    w["cu"] = W.cu_from_lengths(LENGTHS)
    tdt = torch.bfloat16 if dt == W.BF16 else torch.float32
    dev = {key: torch.from_numpy(w[key]).cuda().to(tdt).contiguous() for key in ("q", "k", "v")}
    dev["beta"] = torch.from_numpy(w["beta"]).cuda().contiguous()
    dev["log_alpha"] = torch.from_numpy(w["log_alpha"]).cuda().contiguous()
    return w, dev


def _compare(res, ref, cu, keys, tol, tag, kda_gate=None):
    """Per (segment, head) errors.  With kda_gate the operator is compared as
    T_C and log_decay by its bounds (the KDA cache's scalar split is free)."""
    worst = {key: 0.0 for key in keys}
    if "o" in keys:
        got = _np(res["o"])
        for h in range(4):  # every row, short segments included
            worst["o"] = max(worst["o"], rel(got[:, h], ref["o"][:, h]))
    for s in range(len(cu) - 1):
        lo, hi = int(cu[s]), int(cu[s + 1])
        for h in range(4):
            for key in keys:
                got = _np(res[key])
                if key == "o":
                    e = rel(got[lo:hi, h], ref["o"][lo:hi, h]) if hi > lo else 0.0
                elif kda_gate is not None and key == "P_hat":
                    e = tc_error(got[s, h], _np(res["log_decay"])[s, h], ref["P_hat"][s, h],
                                 ref["log_decay"][s, h])
                elif kda_gate is not None and key == "log_decay":
                    e = 0.0 if check_log_decay(got[s, h], kda_gate[lo:hi, h]) else np.inf
                elif key == "log_decay":
                    e = float(np.max(np.abs(got[s, h] - ref[key][s, h])))
                else:
                    e = rel(got[s, h], ref[key][s, h])
                worst[key] = max(worst[key], e)
    print("%s max err: %s" % (tag, {k: "%.2e" % v for k, v in worst.items()}), flush=True)
    for key, val in worst.items():
        assert val <= tol, (tag, key, val)


@pytest.mark.parametrize("d_k,d_v", DIMS)
@pytest.mark.parametrize("dt", [W.BF16, W.F32])
def test_gdn_build_mixed_dims(hy, d_k, d_v, dt):
    _say("gdn build %s d_k=%d d_v=%d lengths %s" % (dt, d_k, d_v, LENGTHS))
    w, dev = _tokens(d_k, d_v, dt, 41)
    res = hy.build_segment(dev["q"], dev["k"], dev["v"], dev["beta"], dev["log_alpha"], w["cu"])
    torch.cuda.synchronize()
    ref = G.build_segments(w["q"], w["k"], w["v"], w["beta"], w["log_alpha"], w["cu"])
    _compare(res, ref, w["cu"], ("o", "S_seg", "P_hat", "log_decay"), TOL[dt],
             "gdn %s %dx%d" % (dt, d_k, d_v))


@pytest.mark.parametrize("d_k,d_v", DIMS)
@pytest.mark.parametrize("family", ["scalar", "diagonal"])
def test_family_build_mixed_dims(hy, d_k, d_v, family):
    _say("family %s build bf16 d_k=%d d_v=%d lengths %s" % (family, d_k, d_v, LENGTHS))
    w, dev = _tokens(d_k, d_v, W.BF16, 42)
    gate = W.family_gate(family, int(w["cu"][-1]), 4, d_k, 43)
    res = hy.family_build(family, dev["q"], dev["k"], dev["v"], torch.from_numpy(gate).cuda(),
                          w["cu"])
    torch.cuda.synchronize()
    ref = F.family_build_segments(family, w["q"], w["k"], w["v"], gate, w["cu"])
    _compare(res, ref, w["cu"], ("o", "S_seg", "log_decay"), TOL[W.BF16],
             "%s %dx%d" % (family, d_k, d_v))


@pytest.mark.parametrize("d_k,d_v", DIMS)
def test_kda_build_mixed_dims(hy, d_k, d_v):
    _say("kda build bf16 d_k=%d d_v=%d lengths %s" % (d_k, d_v, LENGTHS))
    w, dev = _tokens(d_k, d_v, W.BF16, 44)
    gate = W.family_gate("diagonal", int(w["cu"][-1]), 4, d_k, 45)
    res = hy.kda_build(dev["q"], dev["k"], dev["v"], dev["beta"], torch.from_numpy(gate).cuda(),
                       w["cu"])
    torch.cuda.synchronize()
    ref = K.kda_build_segments(w["q"], w["k"], w["v"], w["beta"], gate, w["cu"])
    _compare(res, ref, w["cu"], ("o", "S_seg", "P_hat", "log_decay"), TOL[W.BF16],
             "kda %dx%d" % (d_k, d_v), kda_gate=gate)


@pytest.mark.parametrize("d_k,d_v", DIMS)
def test_compose_and_rescan_mixed_dims(hy, d_k, d_v):
    """The one-pass composition with seams (Sec. 4.3, Eq. (6)) at unequal
    widths: d_v = 64 leaves two of the four column slots idle (they pass the
    composition's barriers), d_k = 64 stages two output tiles instead of four."""
    import oracle
    _say("compose and rescan bf16 d_k=%d d_v=%d" % (d_k, d_v))
    w, dev = _tokens(d_k, d_v, W.BF16, 46)
    cu = w["cu"]
    res = hy.build_segment(dev["q"], dev["k"], dev["v"], dev["beta"], dev["log_alpha"], cu)
    ids = np.array([1, 0, 2, 1, 2, 0], dtype=np.int32)
    offs = np.array([0, 2, 2, 6], dtype=np.int32)  # the second request is empty
    seam_w = 64
    S_out, o_seam = hy.compose_and_rescan(res["P_hat"], res["log_decay"], res["S_seg"], dev["q"],
                                          dev["k"], dev["v"], dev["beta"], dev["log_alpha"],
                                          cu[:-1], np.diff(cu), seam_w, ids, offs)
    torch.cuda.synchronize()
    P, ld, S = _np(res["P_hat"]), _np(res["log_decay"]), _np(res["S_seg"])
    R_out, R_inc = oracle.compose(P, ld, S, ids, offs)
    R_o, _ = oracle.seam(w["q"], w["k"], w["v"], w["beta"], w["log_alpha"], cu[:-1][ids],
                         np.diff(cu)[ids], seam_w, R_inc)
    So, og = _np(S_out), _np(o_seam)
    ws = max(rel(So[r, h], R_out[r, h]) for r in range(3) for h in range(4))
    wo = 0.0
    for j in range(len(ids)):
        wj = min(seam_w, LENGTHS[ids[j]])
        for h in range(4):
            wo = max(wo, rel(og[j, :wj, h], R_o[j, :wj, h]))
    print("compose and rescan %dx%d: state %.2e, seam outputs %.2e" % (d_k, d_v, ws, wo),
          flush=True)
    assert ws <= 1e-4 and wo <= 1e-2
