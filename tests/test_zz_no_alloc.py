"""hypic_build_segment_noalloc against hypic_build_segment, through the C ABI:
two calls in a row, the second with a smaller input, both with more than 128
segments so that the longest-first order goes through the library's fixed
device array; then a call of at most 128 segments.  Results must be bitwise
equal to the workspace entry point's (the same kernels; the order only
schedules)."""

import ctypes
import sys

import numpy as np
import pytest
import torch

from paper_2607_01299_amd import _lib
from paper_2607_01299_amd import workloads as W

pytestmark = pytest.mark.gpu


def _say(msg):
    print("[case] " + msg, flush=True)
    sys.stdout.flush()


def _p(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _run(lib, entry, w, with_ws):
    dev = torch.device("cuda")
    q, k, v = [torch.from_numpy(w[key]).to(dev).to(torch.bfloat16).contiguous()
               for key in ("q", "k", "v")]
    beta = torch.from_numpy(w["beta"]).to(dev)
    la = torch.from_numpy(w["log_alpha"]).to(dev)
    cu = np.ascontiguousarray(w["cu_seqlens"], dtype=np.int32)
    cu_d = torch.from_numpy(cu).to(dev)
    T, h_qk, d_k = q.shape
    h_v, d_v = v.shape[1:]
    n_seg = len(cu) - 1
    dims = _lib.Dims(h_qk=h_qk, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_lib.HYPIC_BF16, chunk=64)
    o = torch.full((T, h_v, d_v), 5.0, dtype=torch.bfloat16, device=dev)
    S = torch.full((n_seg, h_v, d_k, d_v), 5.0, device=dev)
    P = torch.full((n_seg, h_v, d_k, d_k), 5.0, device=dev)
    ld = torch.full((n_seg, h_v), 5.0, device=dev)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    hcu = cu.ctypes.data_as(ctypes.c_void_p)
    if with_ws:
        need = lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(dims), n_seg)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        code = entry(ctypes.byref(dims), _p(q), _p(k), _p(v), _p(beta), _p(la), T, _p(cu_d),
                     hcu, n_seg, _p(o), _p(S), _p(P), _p(ld), _p(ws), need, stream)
    else:
        code = entry(ctypes.byref(dims), _p(q), _p(k), _p(v), _p(beta), _p(la), T, _p(cu_d),
                     hcu, n_seg, _p(o), _p(S), _p(P), _p(ld), stream)
    torch.cuda.synchronize()
    assert code == _lib.HYPIC_OK, code
    return {"o": o, "S_seg": S, "P_hat": P, "log_decay": ld}


def _workload(n_seg, seed):
    rng = np.random.default_rng(seed)
    lengths = rng.integers(1, 90, size=n_seg)
    return W.segment_workload(2, lengths=lengths, heads=(2, 4), d=64, seed=seed)


def test_noalloc_build_matches_the_workspace_build():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    lib = _lib.load()
    for n_seg, seed in ((300, 71), (150, 72), (100, 73)):
        _say("noalloc build: %d segments (d = 64, heads 2/4, bf16), seed %d" % (n_seg, seed))
        w = _workload(n_seg, seed)
        a = _run(lib, lib.hypic_build_segment_noalloc, w, with_ws=False)
        b = _run(lib, lib.hypic_build_segment, w, with_ws=True)
        for key in ("o", "S_seg", "P_hat", "log_decay"):
            assert torch.equal(a[key], b[key]), (n_seg, key)
        # every output was written (no sentinel left)
        assert not torch.any(a["log_decay"] == 5.0)
