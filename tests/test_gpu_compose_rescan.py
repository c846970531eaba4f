"""Composition with seams in one pass (Sec. 4.3 with whole-segment tuples; the
seam does not advance the state) through hypic_compose_and_rescan: S_out must
be the Eq. (6) composition and o_seam the seam outputs from each incoming
state, against the float64 oracle on the same pool tuples, and against the
two-launch path (hypic_compose_segments, then hypic_seam_rescan on its incoming
states).  Bars: 1e-4 for the composed states (float32 tuples, split-bf16
products), 1e-2 for the bf16 seam outputs."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_01299_amd import workloads as W

from test_gpu_parity import _dev, _np, _say, rel

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hy():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2607_01299_amd as hy
    from paper_2607_01299_amd import _lib
    _lib.load()
    return hy


@pytest.mark.parametrize("d,heads,w", [(128, (2, 4), 64), (64, (2, 2), 8), (128, (1, 2), 37)])
def test_compose_and_rescan_matches_oracle(hy, d, heads, w):
    lens = [200, 40, 1, 130, 64, 20]
    _say("compose and rescan bf16 d=%d heads=%s w=%d lengths %s" % (d, heads, w, lens))
    wl = W.segment_workload(2, lengths=lens, heads=heads, d=d, seed=95)
    dv = _dev(wl)
    cu = wl["cu_seqlens"]
    res = hy.build_segment(dv["q"], dv["k"], dv["v"], dv["beta"], dv["log_alpha"], cu)
    ids = np.array([2, 0, 3, 1, 4, 5, 1, 2, 0, 3], dtype=np.int32)
    offs = np.array([0, 3, 4, 4, 10], dtype=np.int32)  # the third request is empty
    h_v = heads[1]
    rng = np.random.default_rng(96)
    prefix = (rng.standard_normal((4, h_v, d, d)) * 0.2).astype(np.float32)
    S_out, o_seam = hy.compose_and_rescan(res["P_hat"], res["log_decay"], res["S_seg"], dv["q"],
                                          dv["k"], dv["v"], dv["beta"], dv["log_alpha"], cu[:-1],
                                          np.diff(cu), w, ids, offs,
                                          S_prefix=torch.from_numpy(prefix).cuda())
    torch.cuda.synchronize()
    P, ld, S = _np(res["P_hat"]), _np(res["log_decay"]), _np(res["S_seg"])
    R_out, R_inc = oracle.compose(P, ld, S, ids, offs, S_prefix=prefix)
    R_o, _ = oracle.seam(wl["q"], wl["k"], wl["v"], wl["beta"], wl["log_alpha"],
                         cu[:-1][ids], np.diff(cu)[ids], w, R_inc)
    So, og = _np(S_out), _np(o_seam)
    ws = 0.0
    for r in range(4):
        for h in range(h_v):
            ws = max(ws, rel(So[r, h], R_out[r, h]))
    wo = 0.0
    for j in range(len(ids)):
        wj = min(w, lens[ids[j]])
        for h in range(h_v):
            wo = max(wo, rel(og[j, :wj, h], R_o[j, :wj, h]))
    print("max rel err: state %.2e, seam outputs %.2e" % (ws, wo), flush=True)
    assert ws <= 1e-4 and wo <= 1e-2
    assert np.array_equal(So[2], prefix[2])  # an empty request returns its prefix


def test_compose_and_rescan_serve_burst_equals_two_launches(hy):
    """The serve-time burst (256 requests x U{8..64} of the 512-entry pool, w = 64):
    the one-pass call against the composition + seam launches, every output, and
    sampled (request, head) pairs against the oracle."""
    _say("compose and rescan: serve burst against the two-launch path")
    from paper_2607_01299_amd.pipeline import ComposeBurst
    p = W.pool_workload()
    t = p["tokens"]
    toks = (torch.from_numpy(t["q"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["k"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["v"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["beta"]).cuda(), torch.from_numpy(t["log_alpha"]).cuda())
    pool = (torch.from_numpy(p["P_hat"]).cuda(), torch.from_numpy(p["log_decay"]).cuda(),
            torch.from_numpy(p["S_seg"]).cuda())
    two = ComposeBurst(*pool, p["seg_ids"], p["req_offsets"], toks, p["tok_start"], p["tok_len"],
                       p["w"])
    two.run()
    # the composition alone (no incoming states written) gives the same S_out,
    # bit for bit: the same kernel with its incoming-state stores skipped
    S_two = two.S_out.clone()
    two.S_out.fill_(float("nan"))
    two.compose_states()
    torch.cuda.synchronize()
    assert torch.equal(two.S_out, S_two)
    S_out, o_seam = hy.compose_and_rescan(*pool, *toks, p["tok_start_pool"], p["seam_len_pool"],
                                          p["w"], p["seg_ids"], p["req_offsets"])
    torch.cuda.synchronize()
    n_req = len(p["req_offsets"]) - 1
    a, b = _np(S_out), _np(two.S_out)
    worst_s = max(rel(a[r, h], b[r, h]) for r in range(n_req) for h in range(16))
    oa, ob = _np(o_seam), _np(two.o_seam)
    worst_o = max(rel(oa[j, :, h], ob[j, :, h]) for j in range(0, two.nnz, 7) for h in range(16))
    print("one pass vs two launches: state %.2e, seam outputs %.2e" % (worst_s, worst_o),
          flush=True)
    assert worst_s <= 1e-4 and worst_o <= 1e-2
    pairs = [(0, 0), (77, 5), (255, 15)]
    R_out, R_inc = oracle.compose(p["P_hat"], p["log_decay"], p["S_seg"], p["seg_ids"],
                                  p["req_offsets"], req_head_pairs=pairs)
    for r, h in pairs:
        assert rel(a[r, h], R_out[r, h]) <= 1e-4, (r, h)
        j0, j1 = int(p["req_offsets"][r]), int(p["req_offsets"][r + 1])
        R_o, _ = oracle.seam(t["q"], t["k"], t["v"], t["beta"], t["log_alpha"],
                             p["tok_start"][j0:j1], p["tok_len"][j0:j1], 64, R_inc[j0:j1],
                             entry_head_pairs=[(e, h) for e in range(j1 - j0)])
        for e in range(j1 - j0):
            assert rel(oa[j0 + e, :, h], R_o[e, :, h]) <= 1e-2, (r, h, e)
