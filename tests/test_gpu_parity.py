"""Parity of the HIP path (through the C ABI) against the float64 oracle.

Tolerances (relative Frobenius error per (segment, head) tensor, maximum over
all): 1e-4 for float32 inputs, 1e-2 for bf16 inputs with float32 accumulation
(the bf16 bound includes the bf16 rounding of o).  log_decay is compared by its
absolute error, which is the relative error it induces in
P_seg = exp(log_decay) * P_hat.  Every GPU test prints the case it runs before
touching the GPU.
"""

import sys

import numpy as np
import pytest
import torch

import oracle
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


def _dev(w, device="cuda"):
    dt = torch.bfloat16 if w["dtype"] == W.BF16 else torch.float32
    out = {}
    for key in ("q", "k", "v"):
        out[key] = torch.from_numpy(w[key]).to(device).to(dt).contiguous()
    for key in ("beta", "log_alpha"):
        out[key] = torch.from_numpy(w[key]).to(device).contiguous()
    return out


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel(x, ref):
    nr = np.linalg.norm(ref)
    if nr == 0.0:
        return float(np.linalg.norm(x))
    return float(np.linalg.norm(x - ref) / nr)


def _check_build(res, ref, cu, pairs, tol, tag=""):
    """Compare GPU build results with the oracle on the given (segment, head) pairs."""
    o, S, P, ld = (_np(res["o"]), _np(res["S_seg"]),
                   _np(res["P_hat"]) if res["P_hat"] is not None else None,
                   _np(res["log_decay"]) if res["log_decay"] is not None else None)
    worst = {"o": 0.0, "S": 0.0, "P": 0.0, "ld": 0.0}
    for s, h in pairs:
        lo, hi = int(cu[s]), int(cu[s + 1])
        if hi > lo:
            worst["o"] = max(worst["o"], rel(o[lo:hi, h], ref["o"][lo:hi, h]))
        worst["S"] = max(worst["S"], rel(S[s, h], ref["S_seg"][s, h]))
        if P is not None:
            worst["P"] = max(worst["P"], rel(P[s, h], ref["P_hat"][s, h]))
            worst["ld"] = max(worst["ld"], abs(ld[s, h] - ref["log_decay"][s, h]))
            if ref["log_decay"][s, h] > -80.0:
                Pm = np.exp(ld[s, h]) * P[s, h]
                Pr = np.exp(ref["log_decay"][s, h]) * ref["P_hat"][s, h]
                worst["P"] = max(worst["P"], rel(Pm, Pr))
    print("%s max rel err: %s" % (tag, {k: "%.2e" % v for k, v in worst.items()}), flush=True)
    for key, val in worst.items():
        assert val <= tol, (tag, key, val)
    return worst


def _all_pairs(n_seg, h_v):
    return [(s, h) for s in range(n_seg) for h in range(h_v)]


# ---------------------------------------------------------------------------
# configuration 1: float32, one head, d = 64, 4 x 256 tokens
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("chunk", [64, 32, 16])
def test_cfg1_build_compose_seam_fp32(hy, chunk):
    _say("cfg1 fp32 d=64 4x256 chunk=%d: build + compose + seam" % chunk)
    w = W.segment_workload(1)
    d = _dev(w)
    cu = w["cu_seqlens"]
    res = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu, chunk=chunk)
    ids = np.arange(4, dtype=np.int32)
    offs = np.array([0, 4], dtype=np.int32)
    S_out, S_inc = hy.compose_segments(res["P_hat"], res["log_decay"], res["S_seg"], ids, offs,
                                       precision="f32")
    seam_w = 32
    o_seam, S_post = hy.seam_rescan(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"],
                                    cu[:-1], np.diff(cu), seam_w, S_inc, chunk=chunk)
    torch.cuda.synchronize()
    ref = oracle.build_segments(w["q"], w["k"], w["v"], w["beta"], w["log_alpha"], cu)
    _check_build(res, ref, cu, _all_pairs(4, 1), TOL[W.F32], "cfg1 chunk=%d" % chunk)
    R_out, R_inc = oracle.compose(ref["P_hat"], ref["log_decay"], ref["S_seg"], ids, offs)
    assert rel(_np(S_out)[0, 0], R_out[0, 0]) <= TOL[W.F32]
    for j in range(4):
        assert rel(_np(S_inc)[j, 0], R_inc[j, 0]) <= TOL[W.F32]
    # the composed state equals the sequential recurrence over all 1024 tokens
    o_full, S_full = oracle.recurrence(w["q"][:, 0], w["k"][:, 0], w["v"][:, 0],
                                       w["beta"][:, 0], w["log_alpha"][:, 0])
    assert rel(_np(S_out)[0, 0], S_full) <= TOL[W.F32]
    # the seam from the composed incoming state reproduces the full run's outputs
    for j in range(4):
        start = int(cu[j])
        assert rel(_np(o_seam)[j, :, 0], o_full[start:start + seam_w]) <= TOL[W.F32]
        _, S_w = oracle.recurrence(w["q"][:start + seam_w, 0], w["k"][:start + seam_w, 0],
                                   w["v"][:start + seam_w, 0], w["beta"][:start + seam_w, 0],
                                   w["log_alpha"][:start + seam_w, 0])
        assert rel(_np(S_post)[j, 0], S_w) <= TOL[W.F32]


# ---------------------------------------------------------------------------
# ragged bf16 / f32 batches, grouped heads, mixed dims, empty segments
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,dk,dv,heads,chunk", [
    (W.BF16, 128, 128, (2, 4), 64),
    (W.BF16, 64, 64, (1, 1), 32),
    (W.F32, 128, 128, (1, 2), 64),
    (W.F32, 64, 128, (2, 2), 32),
    (W.F32, 128, 64, (1, 1), 16),
    (W.BF16, 128, 64, (2, 2), 16),
])
def test_ragged_build_matches_oracle(hy, dtype, dk, dv, heads, chunk):
    lens = [200, 64, 1, 0, 130, 65]
    _say("ragged build dtype=%s dk=%d dv=%d heads=%s chunk=%d lens=%s"
         % (dtype, dk, dv, heads, chunk, lens))
    w = W.segment_workload(2, lengths=lens, heads=heads, dtype=dtype, d=dk)
    if dk != dv:  # redraw with distinct key / value widths
        rng = np.random.default_rng(7)
        T = int(sum(lens))
        w.update(W.draw_tokens(rng, T, heads[0], heads[1], dk, dv, dtype))
    d = _dev(w)
    cu = w["cu_seqlens"]
    res = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu, chunk=chunk)
    torch.cuda.synchronize()
    ref = oracle.build_segments(w["q"], w["k"], w["v"], w["beta"], w["log_alpha"], cu)
    _check_build(res, ref, cu, _all_pairs(len(lens), heads[1]), TOL[dtype], "ragged")
    # the empty segment carries the identity tuple
    assert np.all(_np(res["S_seg"])[3] == 0)
    assert np.array_equal(_np(res["P_hat"])[3, 0], np.eye(dk))
    assert np.all(_np(res["log_decay"])[3] == 0)


@pytest.mark.parametrize("dtype,d", [(W.BF16, 128), (W.F32, 64)])
def test_many_segments_device_order(hy, dtype, d):
    """Past 128 segments the longest-first order is computed on the device."""
    rng = np.random.default_rng(11)
    lens = [int(x) for x in rng.integers(0, 90, size=160)]
    lens[5] = 0
    _say("many segments dtype=%s d=%d n_seg=%d tokens=%d" % (dtype, d, len(lens), sum(lens)))
    w = W.segment_workload(2, lengths=lens, heads=(1, 2), dtype=dtype, d=d)
    dv = _dev(w)
    cu = w["cu_seqlens"]
    res = hy.build_segment(dv["q"], dv["k"], dv["v"], dv["beta"], dv["log_alpha"], cu)
    torch.cuda.synchronize()
    ref = oracle.build_segments(w["q"], w["k"], w["v"], w["beta"], w["log_alpha"], cu)
    _check_build(res, ref, cu, _all_pairs(len(lens), 2), TOL[dtype], "many segments")


def test_build_is_deterministic_and_batch_independent(hy):
    _say("determinism / batch independence bf16 d=128")
    w = W.segment_workload(2, lengths=[300, 70, 129], heads=(2, 2))
    d = _dev(w)
    cu = w["cu_seqlens"]
    a = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu)
    b = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu)
    lo, hi = int(cu[1]), int(cu[2])
    alone = hy.build_segment(d["q"][lo:hi].contiguous(), d["k"][lo:hi].contiguous(),
                             d["v"][lo:hi].contiguous(), d["beta"][lo:hi].contiguous(),
                             d["log_alpha"][lo:hi].contiguous(), [0, hi - lo])
    torch.cuda.synchronize()
    for key in ("o", "S_seg", "P_hat", "log_decay"):
        assert torch.equal(a[key], b[key]), key
    assert torch.equal(alone["S_seg"][0], a["S_seg"][1])
    assert torch.equal(alone["P_hat"][0], a["P_hat"][1])
    assert torch.equal(alone["o"], a["o"][lo:hi])


def test_grouped_heads_with_equal_gates_share_operator(hy):
    _say("GVA equal gates bf16")
    w = W.segment_workload(3, n_seg=2, seg_len=150, heads=(1, 2))
    w["beta"][:, 1] = w["beta"][:, 0]
    w["log_alpha"][:, 1] = w["log_alpha"][:, 0]
    d = _dev(w)
    res = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], w["cu_seqlens"])
    torch.cuda.synchronize()
    assert torch.equal(res["P_hat"][:, 0], res["P_hat"][:, 1])
    assert not torch.equal(res["S_seg"][:, 0], res["S_seg"][:, 1])


def test_slow_decay_composition_bf16(hy):
    """Slow decay (alpha = 1 - 2^-10, the slowest head of Tab. 2) keeps earlier
    segments visible in the composed state, so operator errors would show."""
    _say("slow-decay compose bf16 d=128 3x256")
    w = W.segment_workload(2, lengths=[256, 256, 256], heads=(1, 1), gate="slow")
    d = _dev(w)
    cu = w["cu_seqlens"]
    res = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu)
    S_out, _ = hy.compose_segments(res["P_hat"], res["log_decay"], res["S_seg"], [0, 1, 2],
                                   [0, 3], want_incoming=False)
    torch.cuda.synchronize()
    _, S_full = oracle.recurrence(w["q"][:, 0], w["k"][:, 0], w["v"][:, 0], w["beta"][:, 0],
                                  w["log_alpha"][:, 0])
    err = rel(_np(S_out)[0, 0], S_full)
    # naive addition would be far off: the composition is doing real work here
    naive = rel(_np(res["S_seg"]).sum(axis=0)[0], S_full)
    print("slow decay: composed err %.2e, naive-addition err %.2e" % (err, naive), flush=True)
    assert err <= TOL[W.BF16] and naive > 0.1


# ---------------------------------------------------------------------------
# composition and seam on a synthetic pool (configuration-5 structure)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("precision", ["split", "f32"])
def test_pool_compose_and_seam(hy, precision):
    _say("pool compose+seam precision=%s" % precision)
    p = W.pool_workload(n_pool=24, n_req=5, n_min=1, n_max=12, heads=2, d=128,
                        seam_tokens=64, w=40)
    dev = "cuda"
    P = torch.from_numpy(p["P_hat"]).to(dev)
    g = torch.from_numpy(p["log_decay"]).to(dev)
    S = torch.from_numpy(p["S_seg"]).to(dev)
    rng = np.random.default_rng(3)
    S_prefix = (rng.standard_normal((5, 2, 128, 128)) * 0.3).astype(np.float32)
    S_out, S_inc = hy.compose_segments(P, g, S, p["seg_ids"], p["req_offsets"],
                                       torch.from_numpy(S_prefix).to(dev), precision=precision)
    tk = _dev(dict(p["tokens"], dtype=W.BF16))
    o_seam, S_post = hy.seam_rescan(tk["q"], tk["k"], tk["v"], tk["beta"], tk["log_alpha"],
                                    p["tok_start"], p["tok_len"], p["w"], S_inc)
    torch.cuda.synchronize()
    R_out, R_inc = oracle.compose(p["P_hat"], p["log_decay"], p["S_seg"], p["seg_ids"],
                                  p["req_offsets"], S_prefix=S_prefix)
    tol = TOL[W.BF16]
    e_out = max(rel(_np(S_out)[r, h], R_out[r, h]) for r in range(5) for h in range(2))
    e_inc = max(rel(_np(S_inc)[j, h], R_inc[j, h]) for j in range(len(p["seg_ids"]))
                for h in range(2))
    t = p["tokens"]
    R_o, R_post = oracle.seam(t["q"], t["k"], t["v"], t["beta"], t["log_alpha"], p["tok_start"],
                              p["tok_len"], p["w"], R_inc)
    e_o = max(rel(_np(o_seam)[j, :, h], R_o[j, :, h]) for j in range(len(p["seg_ids"]))
              for h in range(2))
    e_p = max(rel(_np(S_post)[j, h], R_post[j, h]) for j in range(len(p["seg_ids"]))
              for h in range(2))
    print("pool %s: S_out %.2e S_inc %.2e o_seam %.2e S_post %.2e"
          % (precision, e_out, e_inc, e_o, e_p), flush=True)
    assert max(e_out, e_inc) <= 1e-4       # float32 operands, split or f32 matrix cores
    assert max(e_o, e_p) <= tol


def test_compose_empty_request_returns_prefix(hy):
    _say("compose empty request")
    dev = "cuda"
    P = torch.randn(3, 1, 64, 64, device=dev)
    g = torch.zeros(3, 1, device=dev)
    S = torch.randn(3, 1, 64, 64, device=dev)
    pre = torch.randn(2, 1, 64, 64, device=dev)
    out, inc = hy.compose_segments(P, g, S, [2], [0, 0, 1], pre, precision="f32")
    torch.cuda.synchronize()
    assert torch.equal(out[0], pre[0])
    assert torch.equal(inc[0], pre[1])


@pytest.mark.parametrize("w,dtype", [(8, W.BF16), (40, W.F32), (100, W.BF16)])
def test_seam_widths(hy, w, dtype):
    """w shorter than, longer than and spanning several chunks of a segment."""
    lens = [20, 300, 64, 1]
    _say("seam w=%d dtype=%s lens=%s" % (w, dtype, lens))
    x = W.segment_workload(2, lengths=lens, heads=(1, 2), dtype=dtype)
    d = _dev(x)
    cu = x["cu_seqlens"]
    rng = np.random.default_rng(5)
    S_in = (rng.standard_normal((4, 2, 128, 128)) * 0.3).astype(np.float32)
    o_seam, S_post = hy.seam_rescan(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu[:-1],
                                    np.diff(cu), w, torch.from_numpy(S_in).cuda())
    torch.cuda.synchronize()
    R_o, R_post = oracle.seam(x["q"], x["k"], x["v"], x["beta"], x["log_alpha"], cu[:-1],
                              np.diff(cu), w, S_in)
    tol = TOL[dtype]
    for j, L in enumerate(lens):
        we = min(w, L)
        for h in range(2):
            assert rel(_np(o_seam)[j, :we, h], R_o[j, :we, h]) <= tol, (j, h)
            assert rel(_np(S_post)[j, h], R_post[j, h]) <= tol, (j, h)


def test_error_leaves_outputs_untouched(hy):
    """A rejected call enqueues nothing: a pre-filled output stays as it was."""
    import ctypes
    from paper_2607_01299_amd import _lib
    _say("error path: out-of-range segment id")
    lib = _lib.load()
    dev = "cuda"
    P = torch.zeros(2, 1, 64, 64, device=dev)
    g = torch.zeros(2, 1, device=dev)
    S = torch.zeros(2, 1, 64, 64, device=dev)
    out = torch.full((1, 1, 64, 64), 7.0, device=dev)
    ids = np.array([0, 2], dtype=np.int32)            # 2 is out of range
    offs = np.array([0, 2], dtype=np.int32)
    ids_d = torch.from_numpy(ids).to(dev)
    offs_d = torch.from_numpy(offs).to(dev)
    dims = _lib.Dims(h_qk=1, h_v=1, d_k=64, d_v=64, dtype=_lib.HYPIC_F32, chunk=64)
    code = lib.hypic_compose_segments(
        ctypes.byref(dims), P.data_ptr(), g.data_ptr(), S.data_ptr(), 2, ids_d.data_ptr(),
        ids.ctypes.data_as(ctypes.c_void_p), offs_d.data_ptr(),
        offs.ctypes.data_as(ctypes.c_void_p), 1, None, out.data_ptr(), None, None, 0, None)
    torch.cuda.synchronize()
    assert code == _lib.HYPIC_EINVAL
    assert torch.all(out == 7.0)
    with pytest.raises(hy.HypicError):
        hy.compose_segments(P, g, S, ids, offs)


def test_build_rejects_offsets_past_the_tokens(hy):
    """An offset past the n_tokens rows of q, k, v is rejected on the host: the
    call returns HYPIC_EINVAL and enqueues nothing (pre-filled outputs keep
    their values); the Python layer rejects mismatched tensors before the call."""
    import ctypes
    from paper_2607_01299_amd import _lib
    _say("error path: cu_seqlens past the token arrays, mismatched tensors")
    lib = _lib.load()
    dev = "cuda"
    T, d = 40, 64
    q = torch.zeros(T, 1, d, device=dev, dtype=torch.bfloat16)
    v = torch.zeros(T, 1, d, device=dev, dtype=torch.bfloat16)
    beta = torch.zeros(T, 1, device=dev)
    la = torch.zeros(T, 1, device=dev)
    cu = np.array([0, 20, 48], dtype=np.int32)          # 48 > 40 rows
    cu_d = torch.from_numpy(cu).to(dev)
    o = torch.full((T, 1, d), 3.0, device=dev, dtype=torch.bfloat16)
    S = torch.full((2, 1, d, d), 7.0, device=dev)
    P = torch.full((2, 1, d, d), 7.0, device=dev)
    ld = torch.full((2, 1), 7.0, device=dev)
    dims = _lib.Dims(h_qk=1, h_v=1, d_k=d, d_v=d, dtype=_lib.HYPIC_BF16, chunk=64)
    code = lib.hypic_build_segment(
        ctypes.byref(dims), q.data_ptr(), q.data_ptr(), v.data_ptr(), beta.data_ptr(),
        la.data_ptr(), T, cu_d.data_ptr(), cu.ctypes.data_as(ctypes.c_void_p), 2, o.data_ptr(),
        S.data_ptr(), P.data_ptr(), ld.data_ptr(), None, 0, None)
    torch.cuda.synchronize()
    assert code == _lib.HYPIC_EINVAL
    assert torch.all(o == 3.0) and torch.all(S == 7.0) and torch.all(P == 7.0)
    assert torch.all(ld == 7.0)
    with pytest.raises(hy.HypicError):
        hy.build_segment(q, q, v, beta, la, cu)
    ok = np.array([0, 20, 40], dtype=np.int32)
    with pytest.raises(hy.HypicError):                  # bf16 beta
        hy.build_segment(q, q, v, beta.to(torch.bfloat16), la, ok)
    with pytest.raises(hy.HypicError):                  # float32 v next to bf16 q
        hy.build_segment(q, q, v.float(), beta, la, ok)
    with pytest.raises(hy.HypicError):                  # short incoming states
        hy.seam_rescan(q, q, v, beta, la, [0, 20], [20, 20], 8, S[:1])
    with pytest.raises(hy.HypicError):                  # short P_hat
        hy.compose_segments(P[:1], ld, S, [0, 1], [0, 2])


def test_chain_count_not_a_multiple_of_eight(hy):
    """21 chains x 2 column blocks: the first 16 chains take the XCD-grouped
    workgroup numbering, the last 5 the linear one; both must match the oracle."""
    lens = [97, 130, 64, 1, 200, 33, 150]
    _say("7 segments x 3 v-heads bf16 d=128 lens=%s" % lens)
    w = W.segment_workload(2, lengths=lens, heads=(1, 3))
    d = _dev(w)
    cu = w["cu_seqlens"]
    res = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu)
    torch.cuda.synchronize()
    ref = oracle.build_segments(w["q"], w["k"], w["v"], w["beta"], w["log_alpha"], cu)
    _check_build(res, ref, cu, _all_pairs(len(lens), 3), TOL[W.BF16], "21 chains")


@pytest.mark.parametrize("dk,dv,heads", [(128, 128, (2, 4)), (128, 64, (1, 2)), (64, 128, (1, 1))])
def test_build_without_operator(hy, dk, dv, heads):
    """Without the operator every wave carries state columns; o and S_seg must
    not change."""
    lens = [150, 64, 1, 77]
    _say("build without operator bf16 dk=%d dv=%d heads=%s" % (dk, dv, heads))
    w = W.segment_workload(2, lengths=lens, heads=heads, d=dk)
    if dk != dv:
        rng = np.random.default_rng(11)
        w.update(W.draw_tokens(rng, int(sum(lens)), heads[0], heads[1], dk, dv, W.BF16))
    d = _dev(w)
    cu = w["cu_seqlens"]
    res = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu,
                           want_operator=False)
    full = hy.build_segment(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], cu)
    torch.cuda.synchronize()
    assert res["P_hat"] is None
    ref = oracle.build_segments(w["q"], w["k"], w["v"], w["beta"], w["log_alpha"], cu,
                                want_operator=False)
    worst = 0.0
    for s in range(len(lens)):
        lo, hi = int(cu[s]), int(cu[s + 1])
        for h in range(heads[1]):
            worst = max(worst, rel(_np(res["o"][lo:hi, h]), ref["o"][lo:hi, h]),
                        rel(_np(res["S_seg"][s, h]), ref["S_seg"][s, h]))
    print("no-operator build max rel err %.2e" % worst, flush=True)
    assert worst <= TOL[W.BF16]
    # same arithmetic for the state with or without the operator columns
    assert torch.equal(res["S_seg"], full["S_seg"])
    assert torch.equal(res["o"], full["o"])


def test_graph_replay_matches_eager(hy):
    """The bench's timed step: build, compose and seams captured as one HIP
    graph.  Several replays, with eager work and synchronisations between
    them, reproduce the eager results bit for bit."""
    _say("graph replay vs eager: bf16 16 heads d=128, 3 x 200 tokens")
    from paper_2607_01299_amd.pipeline import SegmentPipeline
    w = W.segment_workload(2, lengths=[200, 77, 130], heads=(4, 8))
    d = _dev(w)
    pipe = SegmentPipeline(d["q"], d["k"], d["v"], d["beta"], d["log_alpha"], w["cu_seqlens"],
                           seam_w=16, want_post=True)
    pipe.run()
    torch.cuda.synchronize()
    outs = ("o", "S_seg", "P_hat", "log_decay", "S_out", "S_inc", "o_seam", "S_post")
    ref = {k: getattr(pipe, k).clone() for k in outs}
    pipe.capture()
    for _ in range(3):
        for k in outs:
            getattr(pipe, k).fill_(-7.0)
        torch.cuda.synchronize()
        pipe.replay()
        torch.cuda.synchronize()
        for k in outs:  # every segment is longer than the seam: all rows are written
            assert torch.equal(getattr(pipe, k), ref[k]), k
        _ = torch.randn(1000, device="cuda").sum().item()  # eager work between replays
