"""Full-size parity: the five workloads at their real sizes, run through the
same pre-bound launches the bench times (SegmentPipeline / ComposeBurst), with
sampled outputs checked against the float64 oracle computed one (segment,
head) at a time.  bf16 tolerance 1e-2 (relative Frobenius per tensor)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_01299_amd import workloads as W

from test_gpu_parity import _np, _say, rel
from _oracle_pool import build_pairs

pytestmark = pytest.mark.gpu

TOL = 1e-2


@pytest.fixture(scope="module")
def pipe_mod():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2607_01299_amd import _lib, pipeline
    _lib.load()
    return pipeline


def _dev(w):
    dt = torch.bfloat16 if w["dtype"] == W.BF16 else torch.float32
    return tuple([torch.from_numpy(w[k]).cuda().to(dt).contiguous() for k in ("q", "k", "v")]
                 + [torch.from_numpy(w[k]).cuda().contiguous() for k in ("beta", "log_alpha")])


def _head(w, h, sl=slice(None)):
    """One v-head (and its qk-head) of a packed batch, as a 1-head problem."""
    h_v, h_qk = w["v"].shape[1], w["q"].shape[1]
    g = oracle.qk_head_of(h, h_v, h_qk)
    return (w["q"][sl, g:g + 1], w["k"][sl, g:g + 1], w["v"][sl, h:h + 1],
            w["beta"][sl, h:h + 1], w["log_alpha"][sl, h:h + 1])


def _spread(n_seg, h_v, extra=()):
    """Every segment once, its head stepping by a stride coprime to h_v, so the
    sample meets every segment, every head, both v-heads of a q/k group and
    both column blocks of every chain (each pair checks all columns); plus
    `extra` pairs."""
    step = 7 if h_v % 7 else 5
    return sorted(set([(s, (step * s + 3) % h_v) for s in range(n_seg)] + list(extra)))


def _check_pairs(pipe, w, pairs):
    cu = w["cu_seqlens"]
    spans = [(int(cu[s]), int(cu[s + 1])) for s, _ in pairs]
    print("  oracle for %d (segment, head) pairs, %d tokens" %
          (len(pairs), sum(hi - lo for lo, hi in spans)), flush=True)
    refs = build_pairs([_head(w, h, slice(lo, hi)) for (s, h), (lo, hi) in zip(pairs, spans)])
    worst = 0.0
    for (s, h), (lo, hi), (o, S, P, ld) in zip(pairs, spans, refs):
        e = max(rel(_np(pipe.o[lo:hi, h]), o), rel(_np(pipe.S_seg[s, h]), S),
                rel(_np(pipe.P_hat[s, h]), P), abs(float(pipe.log_decay[s, h]) - ld))
        print("  seg %d head %d (len %d): %.2e" % (s, h, hi - lo, e), flush=True)
        worst = max(worst, e)
    assert worst <= TOL, worst


def _check_head_chain(pipe, w, h, S_prefix=None, seam_w=None):
    """All segments of one head through the oracle, composed, and seams."""
    cu = w["cu_seqlens"]
    n_seg = len(cu) - 1
    d_k, d_v = w["q"].shape[2], w["v"].shape[2]
    P = np.zeros((n_seg, 1, d_k, d_k))
    S = np.zeros((n_seg, 1, d_k, d_v))
    ld = np.zeros((n_seg, 1))
    for s in range(n_seg):
        lo, hi = int(cu[s]), int(cu[s + 1])
        q, k, v, b, a = _head(w, h, slice(lo, hi))
        _, S[s, 0] = oracle.recurrence(q[:, 0], k[:, 0], v[:, 0], b[:, 0], a[:, 0])
        P[s, 0], ld[s, 0] = oracle.segment_operator(k[:, 0], b[:, 0], a[:, 0])
        if s % 8 == 7 or s == n_seg - 1:
            print("  oracle head %d: %d/%d segments" % (h, s + 1, n_seg), flush=True)
    pre = None if S_prefix is None else S_prefix[:, h:h + 1]
    R_out, R_inc = oracle.compose(P, ld, S, pipe.ids_h, pipe.off_h, S_prefix=pre)
    e_out = rel(_np(pipe.S_out[0, h]), R_out[0, 0])
    e_inc = max(rel(_np(pipe.S_inc[j, h]), R_inc[j, 0]) for j in range(pipe.nnz))
    e_seam = 0.0
    if seam_w is not None:
        R_o, _ = oracle.seam(*_head(w, h), pipe.ts_h, pipe.tl_h, seam_w, R_inc)
        for j in range(pipe.nnz):
            we = min(seam_w, int(pipe.tl_h[j]))
            e_seam = max(e_seam, rel(_np(pipe.o_seam[j, :we, h]), R_o[j, :we, 0]))
    print("  head %d chain: S_out %.2e S_inc %.2e o_seam %.2e" % (h, e_out, e_inc, e_seam),
          flush=True)
    assert max(e_out, e_inc, e_seam) <= TOL


@pytest.mark.timeout(300)
def test_cfg2_full_pipeline(pipe_mod):
    _say("cfg2 full: 16 heads d=128 8x2048 bf16, build+compose+seam(w=8)")
    w = W.segment_workload(2)
    pipe = pipe_mod.SegmentPipeline(*_dev(w), w["cu_seqlens"], seam_w=8)
    pipe.run()
    torch.cuda.synchronize()
    _check_pairs(pipe, w, _spread(8, 16, extra=[(0, 0), (5, 11), (7, 15)]))
    _check_head_chain(pipe, w, 6, seam_w=8)


@pytest.mark.timeout(300)
def test_cfg3_full_pipeline_with_prefix(pipe_mod):
    _say("cfg3 full: 32x4096 bf16, 16 qk / 32 v heads, alpha~U(.9,1), 1024-token prefix")
    w = W.segment_workload(3)
    pre = w["prefix"]
    h_v = w["v"].shape[1]
    # the prefix state: the oracle's zero-start state after the 1024 prefix tokens
    S_prefix = np.zeros((1, h_v, 128, 128), dtype=np.float32)
    for h in range(h_v):
        g = oracle.qk_head_of(h, h_v, w["q"].shape[1])
        _, S = oracle.recurrence(pre["q"][:, g], pre["k"][:, g], pre["v"][:, h],
                                 pre["beta"][:, h], pre["log_alpha"][:, h])
        S_prefix[0, h] = S
    pipe = pipe_mod.SegmentPipeline(*_dev(w), w["cu_seqlens"], seam_w=8,
                                    S_prefix=torch.from_numpy(S_prefix).cuda())
    pipe.run()
    torch.cuda.synchronize()
    _check_pairs(pipe, w, _spread(32, h_v, extra=[(0, 0), (17, 31), (31, 12)]))
    _check_head_chain(pipe, w, 21, S_prefix=S_prefix.astype(np.float64), seam_w=8)


@pytest.mark.timeout(300)
def test_cfg4_full_pipeline_ragged(pipe_mod):
    _say("cfg4 full: 64 log-uniform segments, 16 heads, bf16, seam w=32")
    w = W.segment_workload(4)
    lens = w["lengths"]
    print("  total tokens %d, longest %d, shortest %d" % (lens.sum(), lens.max(), lens.min()),
          flush=True)
    pipe = pipe_mod.SegmentPipeline(*_dev(w), w["cu_seqlens"], seam_w=32)
    pipe.run()
    torch.cuda.synchronize()
    # every third segment (ragged lengths 128..16384) and the extremes
    pairs = [p for p in _spread(len(lens), 16) if p[0] % 3 == 0]
    _check_pairs(pipe, w, sorted(set(pairs + [(int(np.argmax(lens)), 3),
                                              (int(np.argmin(lens)), 9), (40, 14)])))
    _check_head_chain(pipe, w, 10, seam_w=32)


@pytest.mark.timeout(300)
def test_cfg5_full_burst(pipe_mod):
    _say("cfg5 full: 256 requests from a 512-entry fp32 pool, 16 heads, seam w=64")
    p = W.pool_workload()
    t = p["tokens"]
    toks = (torch.from_numpy(t["q"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["k"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["v"]).cuda().to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["beta"]).cuda(), torch.from_numpy(t["log_alpha"]).cuda())
    burst = pipe_mod.ComposeBurst(torch.from_numpy(p["P_hat"]).cuda(),
                                  torch.from_numpy(p["log_decay"]).cuda(),
                                  torch.from_numpy(p["S_seg"]).cuda(), p["seg_ids"],
                                  p["req_offsets"], toks, p["tok_start"], p["tok_len"], p["w"])
    burst.run()
    torch.cuda.synchronize()
    print("  compositions %d" % burst.nnz, flush=True)
    offs = p["req_offsets"]
    worst = 0.0
    for r, h in [(0, 0), (101, 7), (255, 15)]:
        js = np.arange(int(offs[r]), int(offs[r + 1]))
        ids = p["seg_ids"][js]
        R_out, R_inc = oracle.compose(p["P_hat"][:, h:h + 1], p["log_decay"][:, h:h + 1],
                                      p["S_seg"][:, h:h + 1], ids, [0, len(ids)])
        tk = (t["q"][:, h:h + 1], t["k"][:, h:h + 1], t["v"][:, h:h + 1],
              t["beta"][:, h:h + 1], t["log_alpha"][:, h:h + 1])
        R_o, _ = oracle.seam(*tk, p["tok_start"][js], p["tok_len"][js], p["w"], R_inc)
        e = rel(_np(burst.S_out[r, h]), R_out[0, 0])
        for i, j in enumerate(js):
            e = max(e, rel(_np(burst.S_inc[j, h]), R_inc[i, 0]),
                    rel(_np(burst.o_seam[j, :, h]), R_o[i, :, 0]))
        print("  request %d head %d (%d segments): %.2e" % (r, h, len(js), e), flush=True)
        worst = max(worst, e)
    assert worst <= TOL

