"""Parity of the reuse-time steps next to the cache through the C ABI against
the float64 oracle: the RoPE state shift (Eq. (7)), the key re-rotation
(Eq. (8)) and the causal conv with carried state (Sec. 4.2 warm-up).

Tolerances: relative Frobenius error 1e-5 for float32 in and out (the angles
are formed in float64 on both sides), 1e-2 where the output is rounded to
bf16.  Every test prints its case before touching the GPU.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import families as F
from paper_2607_01299_amd import workloads as W

pytestmark = pytest.mark.gpu


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


@pytest.mark.parametrize("d_k,d_v", [(128, 128), (64, 128), (128, 64)])
def test_rope_shift_state(hy, d_k, d_v):
    _say("rope shift state d_k=%d d_v=%d" % (d_k, d_v))
    rng = np.random.default_rng(71)
    n, h = 5, 3
    S = rng.standard_normal((n, h, d_k, d_v)).astype(np.float32)
    delta = np.array([0, 1, -37, 4096, 123457], dtype=np.int32)
    St = torch.from_numpy(S).cuda()
    out = hy.rope_shift_state(St, delta, base=10000.0)
    inplace = St.clone()
    hy.rope_shift_state(inplace, delta, base=10000.0, out=inplace)
    torch.cuda.synchronize()
    o = _np(out)
    assert torch.equal(out, inplace)
    for e in range(n):
        for hh in range(h):
            ref = F.rope_shift_state(S[e, hh], int(delta[e]), 10000.0)
            assert rel(o[e, hh], ref) <= 1e-5, (e, hh)
    assert np.array_equal(o[0], S[0].astype(np.float64))  # delta 0 is the identity


def test_eq7_scalar_family_reuse_with_rope(hy):
    """Scalar-family segments built with their keys rotated from position 0,
    states shifted to their global start (Eq. (7)) and composed (Eq. (6)),
    equal the recurrence over the concatenation with keys at their global
    positions (float32)."""
    lens = [70, 130, 64]
    _say("eq7 reuse: scalar family f32 d=64, lengths %s" % lens)
    base = 10000.0
    w = W.segment_workload(1, lengths=lens, heads=(1, 1), d=64, dtype=W.F32, seed=72)
    cu = w["cu_seqlens"]
    T = int(cu[-1])
    gate = W.family_gate("scalar", T, 1, 64, 73)
    k_local = np.concatenate([F.rope_keys_at(w["k"][cu[s]:cu[s + 1], 0], 0, base)
                              for s in range(3)]).astype(np.float32)[:, None, :]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    res = hy.family_build("scalar", dev(w["q"]), dev(k_local), dev(w["v"]), dev(gate), cu)
    shifted = hy.rope_shift_state(res["S_seg"], cu[:-1].astype(np.int32), base=base)
    S_out, _ = hy.family_compose("scalar", res["log_decay"], shifted, [0, 1, 2], [0, 3])
    torch.cuda.synchronize()
    k_glob = F.rope_keys_at(w["k"][:, 0], 0, base)
    _, S_full = F.family_recurrence("scalar", w["q"][:, 0], k_glob, w["v"][:, 0], gate[:, 0])
    assert rel(_np(S_out)[0, 0], S_full) <= 1e-4


@pytest.mark.parametrize("dt,d", [(W.BF16, 128), (W.F32, 64)])
def test_rope_rerotate_keys(hy, dt, d):
    lens = [100, 0, 1, 257, 64]
    _say("rope re-rotate keys %s d=%d lengths %s" % (dt, d, lens))
    rng = np.random.default_rng(74)
    T, h = sum(lens), 4
    k = rng.standard_normal((T, h, d)).astype(np.float32)
    if dt == W.BF16:
        k = W.round_bf16(k)
    cu = W.cu_from_lengths(lens)
    delta = np.array([5, 7, -3, 99999, 0], dtype=np.int32)
    tdt = torch.bfloat16 if dt == W.BF16 else torch.float32
    kt = torch.from_numpy(k).cuda().to(tdt)
    out = hy.rope_rerotate_keys(kt, cu, delta)
    torch.cuda.synchronize()
    o = _np(out)
    tol = 1e-2 if dt == W.BF16 else 1e-5
    for s in range(len(lens)):
        lo, hi = int(cu[s]), int(cu[s + 1])
        for hh in range(h):
            if hi > lo:
                ref = F.rope_rerotate_keys(k[lo:hi, hh], int(delta[s]), 10000.0)
                assert rel(o[lo:hi, hh], ref) <= tol, (s, hh)


@pytest.mark.parametrize("dt,K,with_state,C", [(W.F32, 4, True, 300), (W.BF16, 4, False, 300),
                                               (W.F32, 1, False, 300), (W.BF16, 8, True, 300),
                                               (W.BF16, 4, True, 2064), (W.F32, 3, True, 1030)])
def test_causal_conv(hy, dt, K, with_state, C):
    lens = [130, 0, 1, 2, 64, 65, 300]
    _say("causal conv %s K=%d state=%s C=%d lengths %s" % (dt, K, with_state, C, lens))
    rng = np.random.default_rng(75)
    T = sum(lens)
    x = rng.standard_normal((T, C)).astype(np.float32)
    if dt == W.BF16:
        x = W.round_bf16(x)
    w = (rng.standard_normal((C, K)) * 0.5).astype(np.float32)
    cu = W.cu_from_lengths(lens)
    n = len(lens)
    st = rng.standard_normal((n, K - 1, C)).astype(np.float32) if with_state else None
    tdt = torch.bfloat16 if dt == W.BF16 else torch.float32
    y, st_out = hy.causal_conv(torch.from_numpy(x).cuda().to(tdt), torch.from_numpy(w).cuda(),
                               cu, None if st is None else torch.from_numpy(st).cuda())
    torch.cuda.synchronize()
    yg, sg = _np(y), _np(st_out)
    tol = 1e-2 if dt == W.BF16 else 1e-5
    for s in range(n):
        lo, hi = int(cu[s]), int(cu[s + 1])
        ref_y, ref_st = F.causal_conv(x[lo:hi], w, conv_state=None if st is None else st[s])
        if hi > lo:
            assert rel(yg[lo:hi], ref_y) <= tol, s
        if K > 1:
            assert np.array_equal(sg[s], ref_st), s  # raw inputs, moved exactly


def test_conv_warmup_through_segments(hy):
    """Segments convolved in one batch, each from the previous one's trailing
    state, reproduce the convolution of the concatenation (float32)."""
    _say("causal conv warm-up chain f32 K=4")
    rng = np.random.default_rng(76)
    lens, C, K = [50, 3, 90], 64, 4
    x = rng.standard_normal((sum(lens), C)).astype(np.float32)
    w = rng.standard_normal((C, K)).astype(np.float32)
    cu = W.cu_from_lengths(lens)
    xt, wt = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    state = None
    ys = []
    for s in range(3):
        part = xt[int(cu[s]):int(cu[s + 1])].contiguous()
        y, state = hy.causal_conv(part, wt, [0, lens[s]], state)
        ys.append(y)
    torch.cuda.synchronize()
    ref, _ = F.causal_conv(x, w)
    assert rel(_np(torch.cat(ys)), ref) <= 1e-5
