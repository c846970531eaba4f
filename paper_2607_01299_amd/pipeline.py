"""Pre-bound passes over the hot path.

``SegmentPipeline``: build every segment of a packed batch, compose the
segments behind an optional prefix (one request in batch order unless a CSR
request list is given), and rescan each listed segment's first w tokens from
its composed incoming state.

``ComposeBurst``: compose many requests from a pool of cached tuples and
rescan the seam of every listed segment.

All outputs, device index arrays and C-ABI arguments are allocated once, so a
call to ``run()`` only enqueues the kernels on the stream that was current at
construction.
"""

import ctypes

import numpy as np
import torch

from . import _checks as C
from . import _lib
from ._lib import Dims


def _i32_pair(x, device):
    h = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
    return h, torch.from_numpy(h.copy()).to(device)


def _p(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _check_tokens_against_pool(tokens, pool_dims, dev):
    """Token arrays (q, k, v, beta, log_alpha) whose heads and widths match the
    pool's (h_v, d_k, d_v) and whose per-token arrays are float32 [T, h_v]."""
    q, k, v, beta, log_alpha = tokens
    T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
    if (h_v, d_k, d_v) != tuple(pool_dims) or q.device != dev:
        C.fail("token arrays (%d heads, %d x %d) do not match the pool (%d heads, %d x %d)"
               % ((h_v, d_k, d_v) + tuple(pool_dims)))
    C.per_token("beta", beta, T, h_v, dev)
    C.per_token("log_alpha", log_alpha, T, h_v, dev)
    return T


def _check_csr(ids_h, off_h):
    if len(off_h) < 1:
        C.fail("req_offsets needs at least one value")
    if int(off_h[-1]) != len(ids_h):
        C.fail("req_offsets[-1] = %d but seg_ids holds %d ids" % (int(off_h[-1]), len(ids_h)))


def _dtype_code(t):
    return _lib.HYPIC_BF16 if t.dtype == torch.bfloat16 else _lib.HYPIC_F32


class SegmentPipeline:
    def __init__(self, q, k, v, beta, log_alpha, cu_seqlens, *, chunk=64, seam_w=8,
                 seg_ids=None, req_offsets=None, S_prefix=None, compose_precision="split",
                 want_post=False):
        self.lib = _lib.load()
        dev = q.device
        self.device = dev
        self.stream = torch.cuda.current_stream(dev)
        sp = ctypes.c_void_p(self.stream.cuda_stream)
        T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
        C.per_token("beta", beta, T, h_v, dev)
        C.per_token("log_alpha", log_alpha, T, h_v, dev)
        self.T, self.h_v, self.d_k, self.d_v = T, h_v, d_k, d_v
        self.dims = Dims(h_qk=h_qk, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_dtype_code(q), chunk=chunk)
        self.cdims = Dims(h_qk=h_v, h_v=h_v, d_k=d_k, d_v=d_v,
                          dtype=_lib.HYPIC_F32 if compose_precision == "f32" else _lib.HYPIC_BF16,
                          chunk=chunk)
        self.inputs = (q, k, v, beta, log_alpha)
        self.cu_h, self.cu_d = _i32_pair(cu_seqlens, dev)
        n_seg = len(self.cu_h) - 1
        self.n_seg = n_seg
        f32 = torch.float32
        self.o = torch.empty((T, h_v, d_v), dtype=q.dtype, device=dev)
        self.S_seg = torch.empty((n_seg, h_v, d_k, d_v), dtype=f32, device=dev)
        self.P_hat = torch.empty((n_seg, h_v, d_k, d_k), dtype=f32, device=dev)
        self.log_decay = torch.empty((n_seg, h_v), dtype=f32, device=dev)
        ws_bytes = self.lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(self.dims),
                                                  n_seg)
        self.ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        self._build_args = (
            ctypes.byref(self.dims), _p(q), _p(k), _p(v), _p(beta), _p(log_alpha), T,
            _p(self.cu_d), self.cu_h.ctypes.data_as(ctypes.c_void_p), n_seg, _p(self.o),
            _p(self.S_seg), _p(self.P_hat), _p(self.log_decay), _p(self.ws), ws_bytes, sp)
        # composition: one request of all segments in batch order by default
        if seg_ids is None:
            seg_ids = np.arange(n_seg, dtype=np.int32)
            req_offsets = np.array([0, n_seg], dtype=np.int32)
        self.ids_h, self.ids_d = _i32_pair(seg_ids, dev)
        self.off_h, self.off_d = _i32_pair(req_offsets, dev)
        _check_csr(self.ids_h, self.off_h)
        n_req = len(self.off_h) - 1
        nnz = int(self.off_h[-1])
        self.n_req, self.nnz = n_req, nnz
        C.state("S_prefix", S_prefix, n_req, h_v, d_k, d_v, dev)
        self.S_prefix = S_prefix
        self.S_out = torch.empty((n_req, h_v, d_k, d_v), dtype=f32, device=dev)
        self.S_inc = torch.empty((nnz, h_v, d_k, d_v), dtype=f32, device=dev)
        self._compose_args = (
            ctypes.byref(self.cdims), _p(self.P_hat), _p(self.log_decay), _p(self.S_seg), n_seg,
            _p(self.ids_d), self.ids_h.ctypes.data_as(ctypes.c_void_p), _p(self.off_d),
            self.off_h.ctypes.data_as(ctypes.c_void_p), n_req, _p(S_prefix), _p(self.S_out),
            _p(self.S_inc), None, 0, sp)
        # seam: the first w tokens of every listed segment
        lens = np.diff(self.cu_h)
        self.seam_w = seam_w
        self.ts_h, self.ts_d = _i32_pair(self.cu_h[:-1][self.ids_h], dev)
        self.tl_h, self.tl_d = _i32_pair(lens[self.ids_h], dev)
        self.o_seam = torch.empty((nnz, seam_w, h_v, d_v), dtype=q.dtype, device=dev)
        self.S_post = (torch.empty((nnz, h_v, d_k, d_v), dtype=f32, device=dev)
                       if want_post else None)
        self._seam_args = (
            ctypes.byref(self.dims), _p(q), _p(k), _p(v), _p(beta), _p(log_alpha), T,
            _p(self.ts_d), _p(self.tl_d), self.ts_h.ctypes.data_as(ctypes.c_void_p),
            self.tl_h.ctypes.data_as(ctypes.c_void_p), nnz, seam_w, _p(self.S_inc),
            _p(self.o_seam), _p(self.S_post), None, 0, sp)

    def build(self):
        _lib.check(self.lib.hypic_build_segment(*self._build_args))

    def compose(self):
        _lib.check(self.lib.hypic_compose_segments(*self._compose_args))

    def seam(self):
        _lib.check(self.lib.hypic_seam_rescan(*self._seam_args))

    def run(self):
        self.build()
        self.compose()
        self.seam()

    def capture(self):
        """Capture build, composition and seams as one HIP graph (replayed by
        replay() on the stream current at that time).  The kernels write no
        memory through memsets, so replays are safe to repeat."""
        self.run()  # first launches (one-time kernel attribute set-up) stay outside
        torch.cuda.synchronize(self.device)
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream(device=self.device)
        side.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.graph(graph, stream=side):
            h = ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream)
            _lib.check(self.lib.hypic_build_segment(*(self._build_args[:-1] + (h,))))
            _lib.check(self.lib.hypic_compose_segments(*(self._compose_args[:-1] + (h,))))
            _lib.check(self.lib.hypic_seam_rescan(*(self._seam_args[:-1] + (h,))))
        torch.cuda.synchronize(self.device)
        self.graph = graph
        return graph

    def replay(self):
        self.graph.replay()


def _deal_requests(seg_ids, req_offsets, lanes):
    """Deal CSR requests over `lanes` groups, longest first (round robin over
    the requests sorted by entry count, ties by index).  Returns per group:
    (request indices in ascending order, its CSR seg_ids, its CSR offsets, the
    caller's CSR rows it holds)."""
    ids = np.ascontiguousarray(np.asarray(seg_ids, dtype=np.int32))
    offs = np.ascontiguousarray(np.asarray(req_offsets, dtype=np.int32))
    lens = np.diff(offs)
    n_req = len(lens)
    lanes = max(1, min(int(lanes), max(n_req, 1)))
    if lanes == 1:
        return [(np.arange(n_req), ids, offs, np.arange(int(offs[-1]) if n_req else 0))]
    order = np.argsort(-lens, kind="stable")
    out = []
    for i in range(lanes):
        grp = np.sort(order[i::lanes])
        rows = np.concatenate([np.arange(offs[r], offs[r + 1]) for r in grp] or
                              [np.zeros(0, np.int64)]).astype(np.int64)
        out.append((grp, ids[rows].astype(np.int32),
                    np.concatenate([[0], np.cumsum(lens[grp])]).astype(np.int32), rows))
    return out


class ComposeBurst:
    """Requests composed from a pool of cached tuples, then seam rescans.
    (Dealing these requests over two streams, as SeamAdvanceBurst can, gains
    about 1 %: both launches fill the whole GPU, so they overlap only at their
    edges.)"""

    def __init__(self, P_hat, log_decay, S_seg, seg_ids, req_offsets, tokens, tok_start,
                 tok_len, w, *, chunk=64, precision="split", want_post=False):
        self.lib = _lib.load()
        dev = S_seg.device
        self.stream = torch.cuda.current_stream(dev)
        sp = ctypes.c_void_p(self.stream.cuda_stream)
        n_pool, h_v, d_k, d_v = C.pool(P_hat, log_decay, S_seg)
        _check_tokens_against_pool(tokens, (h_v, d_k, d_v), dev)
        q, k, v, beta, log_alpha = tokens
        self.tokens = tokens
        self.pool = (P_hat, log_decay, S_seg)
        self.cdims = Dims(h_qk=h_v, h_v=h_v, d_k=d_k, d_v=d_v,
                          dtype=_lib.HYPIC_F32 if precision == "f32" else _lib.HYPIC_BF16,
                          chunk=chunk)
        self.dims = Dims(h_qk=q.shape[1], h_v=h_v, d_k=d_k, d_v=d_v, dtype=_dtype_code(q),
                         chunk=chunk)
        self.ids_h, self.ids_d = _i32_pair(seg_ids, dev)
        self.off_h, self.off_d = _i32_pair(req_offsets, dev)
        _check_csr(self.ids_h, self.off_h)
        n_req = len(self.off_h) - 1
        nnz = int(self.off_h[-1])
        if len(tok_start) != nnz or len(tok_len) != nnz:
            C.fail("tok_start and tok_len must hold one value per listed segment (%d)" % nnz)
        self.n_req, self.nnz, self.h_v, self.d_k, self.d_v = n_req, nnz, h_v, d_k, d_v
        f32 = torch.float32
        self.S_out = torch.empty((n_req, h_v, d_k, d_v), dtype=f32, device=dev)
        self.S_inc = torch.empty((nnz, h_v, d_k, d_v), dtype=f32, device=dev)
        self._compose_args = (
            ctypes.byref(self.cdims), _p(P_hat), _p(log_decay), _p(S_seg), n_pool, _p(self.ids_d),
            self.ids_h.ctypes.data_as(ctypes.c_void_p), _p(self.off_d),
            self.off_h.ctypes.data_as(ctypes.c_void_p), n_req, None, _p(self.S_out),
            _p(self.S_inc), None, 0, sp)
        self.ts_h, self.ts_d = _i32_pair(tok_start, dev)
        self.tl_h, self.tl_d = _i32_pair(tok_len, dev)
        self.w = w
        self.o_seam = torch.empty((nnz, w, h_v, d_v), dtype=q.dtype, device=dev)
        self.S_post = (torch.empty((nnz, h_v, d_k, d_v), dtype=f32, device=dev)
                       if want_post else None)
        self._seam_args = (
            ctypes.byref(self.dims), _p(q), _p(k), _p(v), _p(beta), _p(log_alpha), q.shape[0],
            _p(self.ts_d), _p(self.tl_d), self.ts_h.ctypes.data_as(ctypes.c_void_p),
            self.tl_h.ctypes.data_as(ctypes.c_void_p), nnz, w, _p(self.S_inc), _p(self.o_seam),
            _p(self.S_post), None, 0, sp)

    def compose(self):
        _lib.check(self.lib.hypic_compose_segments(*self._compose_args))

    def compose_states(self):
        """Eq. (6) to S_out alone: the same launch without the incoming states
        (S_incoming = NULL), as a caller that needs no seam issues it."""
        a = list(self._compose_args)
        a[12] = None
        _lib.check(self.lib.hypic_compose_segments(*a))

    def seam(self):
        _lib.check(self.lib.hypic_seam_rescan(*self._seam_args))

    def run(self):
        self.compose()
        self.seam()


class SeamAdvanceBurst:
    """Requests composed from a pool of tail tuples with each entry's seam run
    from the running state first (hypic_compose_with_seams), pre-bound.  With
    advance=False the pool holds whole-segment tuples and each seam runs from
    the state entering its entry without advancing it
    (hypic_compose_and_rescan): the composition and seams of ComposeBurst in
    one pass.

    lanes > 1 splits the requests, dealt longest first, over that many calls on
    streams of their own (default priority).  Each lane then holds its
    requests' S_out and o_seam in its own request order; outputs() assembles
    them in the caller's order.
    """

    def __init__(self, P_hat, log_decay, S_seg, seg_ids, req_offsets, tokens, seam_start,
                 seam_len, w, *, S_prefix=None, lanes=1, advance=True):
        self.entry = "hypic_compose_with_seams" if advance else "hypic_compose_and_rescan"
        self.lib = _lib.load()
        dev = S_seg.device
        self.stream = torch.cuda.current_stream(dev)
        n_pool, h_v, d_k, d_v = C.pool(P_hat, log_decay, S_seg)
        _check_tokens_against_pool(tokens, (h_v, d_k, d_v), dev)
        q, k, v, beta, log_alpha = tokens
        self.tokens = tokens
        self.pool = (P_hat, log_decay, S_seg)
        self.dims = Dims(h_qk=q.shape[1], h_v=h_v, d_k=d_k, d_v=d_v, dtype=_dtype_code(q),
                         chunk=64)
        self.ss_h, self.ss_d = _i32_pair(seam_start, dev)
        self.sl_h, self.sl_d = _i32_pair(seam_len, dev)
        if len(self.ss_h) != n_pool or len(self.sl_h) != n_pool:
            C.fail("seam_start and seam_len must hold one value per pool entry (%d)" % n_pool)
        offs = np.asarray(req_offsets, dtype=np.int32)
        _check_csr(np.asarray(seg_ids), offs)
        n_req = len(offs) - 1
        nnz = int(offs[-1])
        C.state("S_prefix", S_prefix, n_req, h_v, d_k, d_v, dev)
        self.n_req, self.nnz, self.h_v, self.d_k, self.d_v = n_req, nnz, h_v, d_k, d_v
        self.w = int(w)
        self.S_prefix = S_prefix
        self.deal = _deal_requests(seg_ids, req_offsets, lanes)
        lanes = len(self.deal)
        self.groups = [d[0] for d in self.deal]
        self.rows = [d[3] for d in self.deal]
        self.streams = ([self.stream] if lanes == 1 else
                        [torch.cuda.Stream(device=dev) for _ in range(lanes)])
        self.lanes = []
        for (grp, g_ids, g_offs, _), st in zip(self.deal, self.streams):
            g_pre = (S_prefix if (lanes == 1 or S_prefix is None) else
                     S_prefix[torch.as_tensor(grp, device=dev)].contiguous())
            self.lanes.append(self._bind(P_hat, log_decay, S_seg, n_pool, g_ids, g_offs, g_pre,
                                         st, dev))
        self.S_out = self.lanes[0]["S_out"] if lanes == 1 else None
        self.o_seam = self.lanes[0]["o_seam"] if lanes == 1 else None

    def _bind(self, P_hat, log_decay, S_seg, n_pool, ids, offs, S_prefix, stream, dev):
        q, k, v, beta, log_alpha = self.tokens
        ids_h, ids_d = _i32_pair(ids, dev)
        off_h, off_d = _i32_pair(offs, dev)
        n_req = len(off_h) - 1
        nnz = int(off_h[-1])
        max_n = int(np.max(np.diff(off_h))) if n_req > 0 else 0
        S_out = torch.empty((n_req, self.h_v, self.d_k, self.d_v), dtype=torch.float32,
                            device=dev)
        o_seam = torch.empty((nnz, self.w, self.h_v, self.d_v), dtype=q.dtype, device=dev)
        if self.entry == "hypic_compose_with_seams":
            need = self.lib.hypic_seam_compose_workspace_bytes(ctypes.byref(self.dims), n_req,
                                                               max_n)
        else:
            need = self.lib.hypic_workspace_bytes(_lib.HYPIC_OP_COMPOSE_RESCAN,
                                                  ctypes.byref(self.dims), n_req)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        args = (
            ctypes.byref(self.dims), _p(P_hat), _p(log_decay), _p(S_seg), n_pool, _p(q), _p(k),
            _p(v), _p(beta), _p(log_alpha), q.shape[0], _p(self.ss_d),
            self.ss_h.ctypes.data_as(ctypes.c_void_p), _p(self.sl_d),
            self.sl_h.ctypes.data_as(ctypes.c_void_p), self.w, _p(ids_d),
            ids_h.ctypes.data_as(ctypes.c_void_p), _p(off_d),
            off_h.ctypes.data_as(ctypes.c_void_p), n_req, _p(S_prefix), _p(S_out),
            _p(o_seam), _p(ws), need, ctypes.c_void_p(stream.cuda_stream))
        return {"S_out": S_out, "o_seam": o_seam, "ws": ws, "keep": (ids_h, ids_d, off_h, off_d,
                                                                   S_prefix), "args": args}

    def run(self):
        call = getattr(self.lib, self.entry)
        if len(self.lanes) == 1:
            _lib.check(call(*self.lanes[0]["args"]))
            return
        start = torch.cuda.Event()
        start.record(self.stream)
        for lane, st in zip(self.lanes, self.streams):
            st.wait_event(start)
            _lib.check(call(*lane["args"]))
        for st in self.streams:
            done = torch.cuda.Event()
            done.record(st)
            self.stream.wait_event(done)

    def outputs(self):
        """(S_out, o_seam) in the caller's request and CSR order (copies when
        lanes > 1), on the burst's stream."""
        if len(self.lanes) == 1:
            return self.S_out, self.o_seam
        dev = self.lanes[0]["S_out"].device
        S_out = torch.empty((self.n_req, self.h_v, self.d_k, self.d_v), dtype=torch.float32,
                            device=dev)
        o_seam = torch.empty((self.nnz, self.w, self.h_v, self.d_v),
                             dtype=self.lanes[0]["o_seam"].dtype, device=dev)
        for lane, grp, rows in zip(self.lanes, self.groups, self.rows):
            S_out[torch.as_tensor(grp, device=dev)] = lane["S_out"]
            o_seam[torch.as_tensor(rows, device=dev)] = lane["o_seam"]
        return S_out, o_seam


class FamilyPipeline:
    """Scalar- or diagonal-family build, composition of the batch's segments in
    order (one request, or the CSR lists given) and seam rescan, pre-bound."""

    def __init__(self, family, q, k, v, gate, cu_seqlens, *, seam_w=8, seg_ids=None,
                 req_offsets=None, S_prefix=None, want_post=False):
        from .ops import FAMILIES
        self.lib = _lib.load()
        self.family = FAMILIES[family]
        dev = q.device
        self.stream = torch.cuda.current_stream(dev)
        sp = ctypes.c_void_p(self.stream.cuda_stream)
        T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
        C.per_token("gate", gate, T, h_v, dev, None if family == "scalar" else d_k)
        self.T, self.h_v, self.d_k, self.d_v = T, h_v, d_k, d_v
        self.dims = Dims(h_qk=h_qk, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_dtype_code(q), chunk=64)
        self.cdims = Dims(h_qk=h_v, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_lib.HYPIC_F32, chunk=64)
        self.inputs = (q, k, v, gate)
        self.cu_h, self.cu_d = _i32_pair(cu_seqlens, dev)
        n_seg = len(self.cu_h) - 1
        self.n_seg = n_seg
        f32 = torch.float32
        self.o = torch.empty((T, h_v, d_v), dtype=q.dtype, device=dev)
        self.S_seg = torch.empty((n_seg, h_v, d_k, d_v), dtype=f32, device=dev)
        ld_shape = (n_seg, h_v) if family == "scalar" else (n_seg, h_v, d_k)
        self.log_decay = torch.empty(ld_shape, dtype=f32, device=dev)
        ws_bytes = self.lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(self.dims),
                                                  n_seg)
        self.ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        self._build_args = (
            ctypes.byref(self.dims), self.family, _p(q), _p(k), _p(v), _p(gate), T, _p(self.cu_d),
            self.cu_h.ctypes.data_as(ctypes.c_void_p), n_seg, _p(self.o), _p(self.S_seg),
            _p(self.log_decay), _p(self.ws), ws_bytes, sp)
        if seg_ids is None:
            seg_ids = np.arange(n_seg, dtype=np.int32)
            req_offsets = np.array([0, n_seg], dtype=np.int32)
        self.ids_h, self.ids_d = _i32_pair(seg_ids, dev)
        self.off_h, self.off_d = _i32_pair(req_offsets, dev)
        _check_csr(self.ids_h, self.off_h)
        n_req = len(self.off_h) - 1
        nnz = int(self.off_h[-1])
        self.n_req, self.nnz = n_req, nnz
        C.state("S_prefix", S_prefix, n_req, h_v, d_k, d_v, dev)
        self.S_prefix = S_prefix
        self.S_out = torch.empty((n_req, h_v, d_k, d_v), dtype=f32, device=dev)
        self.S_inc = torch.empty((nnz, h_v, d_k, d_v), dtype=f32, device=dev)
        self._compose_args = (
            ctypes.byref(self.cdims), self.family, _p(self.log_decay), _p(self.S_seg), n_seg,
            _p(self.ids_d), self.ids_h.ctypes.data_as(ctypes.c_void_p), _p(self.off_d),
            self.off_h.ctypes.data_as(ctypes.c_void_p), n_req, _p(S_prefix), _p(self.S_out),
            _p(self.S_inc), None, 0, sp)
        lens = np.diff(self.cu_h)
        self.seam_w = seam_w
        self.ts_h, self.ts_d = _i32_pair(self.cu_h[:-1][self.ids_h], dev)
        self.tl_h, self.tl_d = _i32_pair(lens[self.ids_h], dev)
        self.o_seam = torch.empty((nnz, seam_w, h_v, d_v), dtype=q.dtype, device=dev)
        self.S_post = (torch.empty((nnz, h_v, d_k, d_v), dtype=f32, device=dev)
                       if want_post else None)
        self._seam_args = (
            ctypes.byref(self.dims), self.family, _p(q), _p(k), _p(v), _p(gate), T,
            _p(self.ts_d), _p(self.tl_d), self.ts_h.ctypes.data_as(ctypes.c_void_p),
            self.tl_h.ctypes.data_as(ctypes.c_void_p), nnz, seam_w, _p(self.S_inc),
            _p(self.o_seam), _p(self.S_post), None, 0, sp)

    def build(self):
        _lib.check(self.lib.hypic_family_build(*self._build_args))

    def compose(self):
        _lib.check(self.lib.hypic_family_compose(*self._compose_args))

    def seam(self):
        _lib.check(self.lib.hypic_family_seam(*self._seam_args))

    def run(self):
        self.build()
        self.compose()
        self.seam()


class KdaPipeline:
    """KDA build (Tab. 1 KDA row: o, S_seg and the operator tuple), pre-bound;
    the tuples compose with hypic_compose_segments."""

    def __init__(self, q, k, v, beta, gate, cu_seqlens, *, want_operator=True):
        self.lib = _lib.load()
        dev = q.device
        self.stream = torch.cuda.current_stream(dev)
        sp = ctypes.c_void_p(self.stream.cuda_stream)
        T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
        C.per_token("beta", beta, T, h_v, dev)
        C.per_token("gate", gate, T, h_v, dev, d_k)
        self.dims = Dims(h_qk=h_qk, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_dtype_code(q), chunk=64)
        self.inputs = (q, k, v, beta, gate)
        self.cu_h, self.cu_d = _i32_pair(cu_seqlens, dev)
        n_seg = len(self.cu_h) - 1
        f32 = torch.float32
        self.o = torch.empty((T, h_v, d_v), dtype=q.dtype, device=dev)
        self.S_seg = torch.empty((n_seg, h_v, d_k, d_v), dtype=f32, device=dev)
        self.P_hat = (torch.empty((n_seg, h_v, d_k, d_k), dtype=f32, device=dev)
                      if want_operator else None)
        self.log_decay = (torch.empty((n_seg, h_v), dtype=f32, device=dev)
                          if want_operator else None)
        ws_bytes = self.lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(self.dims),
                                                  n_seg)
        self.ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        self._build_args = (
            ctypes.byref(self.dims), _p(q), _p(k), _p(v), _p(beta), _p(gate), T, _p(self.cu_d),
            self.cu_h.ctypes.data_as(ctypes.c_void_p), n_seg, _p(self.o), _p(self.S_seg),
            _p(self.P_hat), _p(self.log_decay), _p(self.ws), ws_bytes, sp)

    def build(self):
        _lib.check(self.lib.hypic_kda_build(*self._build_args))


class FamilyComposeBurst:
    """Many requests composed from a pool of scalar- or diagonal-family
    tuples (Eq. (6) with the compressed operators of Tab. 3), pre-bound."""

    def __init__(self, family, log_decay, S_seg, seg_ids, req_offsets):
        from .ops import FAMILIES
        self.lib = _lib.load()
        self.family = FAMILIES[family]
        dev = S_seg.device
        self.stream = torch.cuda.current_stream(dev)
        sp = ctypes.c_void_p(self.stream.cuda_stream)
        if not isinstance(S_seg, torch.Tensor) or S_seg.dim() != 4:
            C.fail("S_seg must be a 4-d torch tensor")
        n_pool, h_v, d_k, d_v = C.pool(None, log_decay, S_seg,
                                       None if family == "scalar" else S_seg.shape[2])
        self.pool = (log_decay, S_seg)
        self.cdims = Dims(h_qk=h_v, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_lib.HYPIC_F32, chunk=64)
        self.ids_h, self.ids_d = _i32_pair(seg_ids, dev)
        self.off_h, self.off_d = _i32_pair(req_offsets, dev)
        _check_csr(self.ids_h, self.off_h)
        n_req = len(self.off_h) - 1
        nnz = int(self.off_h[-1])
        self.n_req, self.nnz, self.h_v, self.d_k, self.d_v = n_req, nnz, h_v, d_k, d_v
        f32 = torch.float32
        self.S_out = torch.empty((n_req, h_v, d_k, d_v), dtype=f32, device=dev)
        self.S_inc = torch.empty((nnz, h_v, d_k, d_v), dtype=f32, device=dev)
        self._compose_args = (
            ctypes.byref(self.cdims), self.family, _p(log_decay), _p(S_seg), n_pool,
            _p(self.ids_d), self.ids_h.ctypes.data_as(ctypes.c_void_p), _p(self.off_d),
            self.off_h.ctypes.data_as(ctypes.c_void_p), n_req, None, _p(self.S_out),
            _p(self.S_inc), None, 0, sp)

    def compose(self):
        _lib.check(self.lib.hypic_family_compose(*self._compose_args))
