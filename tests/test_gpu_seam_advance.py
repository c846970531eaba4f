"""Reuse with seam windows that advance the state (Sec. 4.3) through
hypic_compose_with_seams, against the float64 oracle: tail tuples built on the
GPU over [w, L), seams run from the running state, then Eq. (4).  The composed
state must also equal the recurrence over each request's concatenated
segments.  Tolerances as in the other parity tests (1e-4 float32, 1e-2 bf16).
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_01299_amd import workloads as W

from test_gpu_parity import _dev, _np, _say, rel

pytestmark = pytest.mark.gpu

TOL = {W.F32: 1e-4, W.BF16: 1e-2}


@pytest.fixture(scope="module")
def hy():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2607_01299_amd as hy
    from paper_2607_01299_amd import _lib
    _lib.load()
    return hy


def _split_offsets(cu, w):
    """Each segment split into its seam part and its tail part, as consecutive
    build segments: [start, start + w_i), [start + w_i, end)."""
    out = [0]
    for s in range(len(cu) - 1):
        lo, hi = int(cu[s]), int(cu[s + 1])
        out += [lo + min(w, hi - lo), hi]
    return np.array(out, dtype=np.int32)


@pytest.mark.parametrize("dt,d,heads,w", [(W.BF16, 128, (2, 4), 32), (W.F32, 64, (1, 2), 16),
                                          (W.BF16, 64, (2, 2), 80)])
def test_compose_with_seams_matches_oracle(hy, dt, d, heads, w):
    lens = [200, 40, 130, 20, 64]
    _say("compose with seams %s d=%d heads=%s w=%d lengths %s" % (dt, d, heads, w, lens))
    wl = W.segment_workload(2, lengths=lens, heads=heads, d=d, dtype=dt, seed=93)
    dv = _dev(wl)
    cu = wl["cu_seqlens"]
    parts = _split_offsets(cu, w)
    res = hy.build_segment(dv["q"], dv["k"], dv["v"], dv["beta"], dv["log_alpha"], parts)
    P = res["P_hat"][1::2].contiguous()
    ld = res["log_decay"][1::2].contiguous()
    S = res["S_seg"][1::2].contiguous()
    ids = np.array([2, 0, 3, 1, 4, 1, 2, 0, 3], dtype=np.int32)
    offs = np.array([0, 3, 4, 4, 9], dtype=np.int32)  # the third request is empty
    h_v = heads[1]
    rng = np.random.default_rng(94)
    prefix = (rng.standard_normal((4, h_v, d, d)) * 0.2).astype(np.float32)
    S_out, o_seam = hy.compose_with_seams(P, ld, S, dv["q"], dv["k"], dv["v"], dv["beta"],
                                          dv["log_alpha"], cu[:-1], np.diff(cu), w, ids, offs,
                                          S_prefix=torch.from_numpy(prefix).cuda())
    torch.cuda.synchronize()
    # the oracle's own tail tuples and its seam-advancing composition
    ref = oracle.build_segments(wl["q"], wl["k"], wl["v"], wl["beta"], wl["log_alpha"], parts)
    R_out, R_o, _ = oracle.compose_with_seams(
        ref["P_hat"][1::2], ref["log_decay"][1::2], ref["S_seg"][1::2], wl["q"], wl["k"], wl["v"],
        wl["beta"], wl["log_alpha"], cu[:-1], np.diff(cu), w, ids, offs, S_prefix=prefix)
    tol = TOL[dt]
    So, og = _np(S_out), _np(o_seam)
    worst = 0.0
    for r in range(4):
        for h in range(h_v):
            worst = max(worst, rel(So[r, h], R_out[r, h]))
    for j in range(len(ids)):
        wj = min(w, lens[ids[j]])
        for h in range(h_v):
            worst = max(worst, rel(og[j, :wj, h], R_o[j, :wj, h]))
    print("max rel err %.2e" % worst, flush=True)
    assert worst <= tol
    # the empty request returns its prefix; reading A equals the concatenation
    assert np.array_equal(So[2], prefix[2])
    g = oracle.qk_head_of(1, h_v, heads[0])
    idx = np.concatenate([np.arange(cu[i], cu[i + 1]) for i in ids[offs[3]:offs[4]]])
    _, S_full = oracle.recurrence(wl["q"][idx, g], wl["k"][idx, g], wl["v"][idx, 1],
                                  wl["beta"][idx, 1], wl["log_alpha"][idx, 1], S0=prefix[3, 1])
    assert rel(So[3, 1], S_full) <= tol


def test_compose_with_seams_serve_burst(hy):
    """The serve-time burst with seams that advance the state: 256 requests x
    U{8..64} entries of the 512-entry pool (its tuples read as tail tuples),
    w = 64, sampled (request, head) pairs against the oracle."""
    _say("compose with seams: serve burst, sampled pairs")
    from paper_2607_01299_amd.pipeline import SeamAdvanceBurst
    p = W.pool_workload()
    t = p["tokens"]
    toks = (torch.from_numpy(t["q"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["k"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["v"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["beta"]).cuda(), torch.from_numpy(t["log_alpha"]).cuda())
    seam_start = (np.arange(p["n_pool"]) * 64).astype(np.int32)
    seam_len = np.full(p["n_pool"], 64, dtype=np.int32)
    burst = SeamAdvanceBurst(torch.from_numpy(p["P_hat"]).cuda(),
                             torch.from_numpy(p["log_decay"]).cuda(),
                             torch.from_numpy(p["S_seg"]).cuda(), p["seg_ids"], p["req_offsets"],
                             toks, seam_start, seam_len, 64)
    burst.run()
    torch.cuda.synchronize()
    pairs = [(0, 0), (77, 5), (255, 15), (130, 9)]
    R_out, R_o, _ = oracle.compose_with_seams(
        p["P_hat"], p["log_decay"], p["S_seg"], t["q"], t["k"], t["v"], t["beta"],
        t["log_alpha"], seam_start, seam_len, 64, p["seg_ids"], p["req_offsets"],
        req_head_pairs=pairs)
    So = _np(burst.S_out)
    worst = 0.0
    for r, h in pairs:
        worst = max(worst, rel(So[r, h], R_out[r, h]))
        for j in range(int(p["req_offsets"][r]), int(p["req_offsets"][r + 1])):
            worst = max(worst, rel(_np(burst.o_seam[j, :, h]), R_o[j, :, h]))
    print("max rel err %.2e" % worst, flush=True)
    assert worst <= TOL[W.BF16]


def test_compose_with_seams_two_lanes_equal_one_call(hy):
    """The serve burst split over two calls on two streams (requests dealt
    longest first) gives exactly the single call's S_out and o_seam, behind a
    prefix state, once the lanes' outputs are put back in request order."""
    _say("compose with seams: serve burst, two lanes against one call")
    from paper_2607_01299_amd.pipeline import SeamAdvanceBurst
    p = W.pool_workload()
    t = p["tokens"]
    toks = (torch.from_numpy(t["q"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["k"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["v"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["beta"]).cuda(), torch.from_numpy(t["log_alpha"]).cuda())
    seam_start = (np.arange(p["n_pool"]) * 64).astype(np.int32)
    seam_len = np.full(p["n_pool"], 64, dtype=np.int32)
    pool = (torch.from_numpy(p["P_hat"]).cuda(), torch.from_numpy(p["log_decay"]).cuda(),
            torch.from_numpy(p["S_seg"]).cuda())
    n_req = len(p["req_offsets"]) - 1
    prefix = torch.randn((n_req, 16, 128, 128), generator=torch.Generator().manual_seed(9)).cuda()
    one = SeamAdvanceBurst(*pool, p["seg_ids"], p["req_offsets"], toks, seam_start, seam_len, 64,
                           S_prefix=prefix)
    two = SeamAdvanceBurst(*pool, p["seg_ids"], p["req_offsets"], toks, seam_start, seam_len, 64,
                           S_prefix=prefix, lanes=2)
    one.run()
    two.run()
    two.run()  # a second run on the same bindings
    S2, o2 = two.outputs()
    torch.cuda.synchronize()
    assert torch.equal(one.S_out, S2)
    assert torch.equal(one.o_seam, o2)
