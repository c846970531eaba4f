"""Edge cases of the pipelined scalar and diagonal family builds (bf16,
d_k = 128: the kernels that stage rows through loader waves and split the
chunk's score tiles among producer waves), through the C ABI against the
float64 oracle and closed forms of the Tab. 1 recurrences:

* one batch mixing an empty segment, one token, one token short of a chunk,
  exactly one chunk, one token past it and several chunks (every tail of the
  staging and masking paths);
* zero gates: no decay, so log_decay is exactly zero and the state is the
  plain sum of k_t v_t^T;
* the strongest per-token decay the 16-token tile references take (-5 on
  every channel, 80 over a tile): finite, and the oracle's outputs;
* 150 segments, past the 128 whose longest-first order travels in the kernel
  arguments (the order is then ranked on the device);
* no outputs requested (o = NULL): the state and log_decay unchanged bit for
  bit.
"""

import numpy as np
import pytest
import torch

from oracle import families as F
from paper_2607_01299_amd import workloads as W

from test_gpu_family import _np, _say, rel

pytestmark = pytest.mark.gpu

TOL = 1e-2


@pytest.fixture(scope="module")
def hy():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2607_01299_amd as hy
    from paper_2607_01299_amd import _lib
    _lib.load()
    return hy


def _run(hy, family, lengths, gate_fn, seed, d_v=128):
    """Build bf16 tokens of the given segment lengths (2 q/k heads, 4 v-heads,
    d_k = 128) with gates from gate_fn(T, h_v) and return the GPU result, the
    float64 inputs the oracle sees and the offsets."""
    rng = np.random.default_rng(seed)
    T = int(sum(lengths))
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    h_qk, h_v, d_k = 2, 4, 128
    q = rng.standard_normal((T, h_qk, d_k)) / np.sqrt(d_k)
    k = rng.standard_normal((T, h_qk, d_k))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, h_v, d_v))
    dev, host = {}, {}
    for name, x in (("q", q), ("k", k), ("v", v)):
        t = torch.from_numpy(x.astype(np.float32)).cuda().to(torch.bfloat16).contiguous()
        dev[name] = t
        host[name] = t.float().cpu().numpy().astype(np.float64)
    gate = gate_fn(T, h_v).astype(np.float32)
    res = hy.family_build(family, dev["q"], dev["k"], dev["v"],
                          torch.from_numpy(gate).cuda().contiguous(), cu)
    torch.cuda.synchronize()
    return res, host, gate.astype(np.float64), cu


def _check(res, ref, cu, tag):
    o, S, ld = _np(res["o"]), _np(res["S_seg"]), _np(res["log_decay"])
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S)) and np.all(np.isfinite(ld)), tag
    worst = {"o": 0.0, "S": 0.0, "ld": 0.0}
    for s in range(len(cu) - 1):
        lo, hi = int(cu[s]), int(cu[s + 1])
        for h in range(S.shape[1]):
            if hi > lo:
                worst["o"] = max(worst["o"], rel(o[lo:hi, h], ref["o"][lo:hi, h]))
            worst["S"] = max(worst["S"], rel(S[s, h], ref["S_seg"][s, h]))
            worst["ld"] = max(worst["ld"],
                              float(np.max(np.abs(ld[s, h] - ref["log_decay"][s, h]))))
    print("%s: %s" % (tag, {k: "%.2e" % v for k, v in worst.items()}), flush=True)
    assert worst["o"] <= TOL and worst["S"] <= TOL and worst["ld"] <= 1e-3, (tag, worst)


@pytest.mark.parametrize("family", ["scalar", "diagonal"])
@pytest.mark.parametrize("d_v", [64, 128])
def test_segment_tails(hy, family, d_v):
    lengths = [130, 0, 1, 63, 64, 65, 300]
    _say("family %s bf16 d_k=128 d_v=%d pipelined build, lengths %s" % (family, d_v, lengths))

    def gate_fn(T, h_v):
        return W.family_gate(family, T, h_v, 128, 91)

    res, host, gate, cu = _run(hy, family, lengths, gate_fn, 31, d_v=d_v)
    ref = F.family_build_segments(family, host["q"], host["k"], host["v"], gate, cu)
    _check(res, ref, cu, "%s d_v=%d tails" % (family, d_v))
    # the empty segment: zero state, zero log_decay
    S, ld = _np(res["S_seg"]), _np(res["log_decay"])
    assert np.count_nonzero(S[1]) == 0 and np.count_nonzero(ld[1]) == 0


@pytest.mark.parametrize("family", ["scalar", "diagonal"])
def test_zero_gates_sum_the_writes(hy, family):
    lengths = [200, 77]
    _say("family %s bf16 zero gates, lengths %s" % (family, lengths))

    def gate_fn(T, h_v):
        return np.zeros((T, h_v) if family == "scalar" else (T, h_v, 128))

    res, host, gate, cu = _run(hy, family, lengths, gate_fn, 32)
    assert np.count_nonzero(_np(res["log_decay"])) == 0
    S = _np(res["S_seg"])
    for s in range(len(lengths)):
        lo, hi = int(cu[s]), int(cu[s + 1])
        for h in range(4):
            kh = host["k"][lo:hi, h // 2]
            closed = kh.T @ host["v"][lo:hi, h]  # no decay: S = sum_t k_t v_t^T
            assert rel(S[s, h], closed) <= TOL, (family, s, h)
    ref = F.family_build_segments(family, host["q"], host["k"], host["v"], gate, cu)
    _check(res, ref, cu, "%s zero gates" % family)


def test_diagonal_strongest_decay(hy):
    lengths = [257, 64]
    _say("family diagonal bf16, gate -5 on every channel, lengths %s" % lengths)

    def gate_fn(T, h_v):
        return np.full((T, h_v, 128), -5.0)

    res, host, gate, cu = _run(hy, "diagonal", lengths, gate_fn, 33)
    ref = F.family_build_segments("diagonal", host["q"], host["k"], host["v"], gate, cu)
    _check(res, ref, cu, "diagonal gate -5")


@pytest.mark.parametrize("family", ["scalar", "diagonal"])
def test_more_segments_than_the_inline_order(hy, family):
    """150 segments: past 128 the longest-first order is ranked on the device
    into the workspace instead of travelling in the kernel arguments; every
    (segment, head) must still land on its own rows."""
    rng = np.random.default_rng(35)
    lengths = [int(x) for x in rng.integers(0, 131, size=150)]
    lengths[7] = 0
    lengths[100] = 130
    _say("family %s bf16 d_k=128, %d segments (%d tokens)" % (family, len(lengths), sum(lengths)))

    def gate_fn(T, h_v):
        return W.family_gate(family, T, h_v, 128, 92)

    res, host, gate, cu = _run(hy, family, lengths, gate_fn, 36)
    ref = F.family_build_segments(family, host["q"], host["k"], host["v"], gate, cu)
    _check(res, ref, cu, "%s 150 segments" % family)


@pytest.mark.parametrize("family", ["scalar", "diagonal"])
def test_without_outputs(hy, family):
    """o = NULL: the build skips the output stores only; S_seg and log_decay
    are bit for bit those of the build that writes o."""
    lengths = [190, 1, 64]
    _say("family %s bf16 d_k=128 without outputs, lengths %s" % (family, lengths))
    rng = np.random.default_rng(37)
    T = int(sum(lengths))
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    q, k, v = [torch.from_numpy(rng.standard_normal(s).astype(np.float32)).cuda()
               .to(torch.bfloat16).contiguous() for s in ((T, 2, 128), (T, 2, 128), (T, 4, 128))]
    gate = torch.from_numpy(W.family_gate(family, T, 4, 128, 93)).cuda().contiguous()
    full = hy.family_build(family, q, k, v, gate, cu)
    bare = hy.family_build(family, q, k, v, gate, cu, want_o=False)
    torch.cuda.synchronize()
    assert bare["o"] is None
    assert torch.equal(full["S_seg"], bare["S_seg"])
    assert torch.equal(full["log_decay"], bare["log_decay"])
