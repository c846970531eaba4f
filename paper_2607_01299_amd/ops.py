"""PyTorch-facing calls of the C ABI: allocate outputs with torch on the
inputs' device, pass raw pointers and the current HIP stream, raise on error.

Index arrays (cu_seqlens, seg_ids, req_offsets, tok_start, tok_len) are given
as host int32 arrays (numpy / list / CPU tensor) and, optionally, as device
int32 tensors holding the same values; when the device copy is omitted it is
made here with a synchronous copy.
"""

import ctypes

import numpy as np
import torch

from . import _checks as C
from . import _lib
from ._lib import Dims, HypicError  # noqa: F401

_ws_cache = {}


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return _lib.HYPIC_BF16
    if t.dtype == torch.float32:
        return _lib.HYPIC_F32
    raise HypicError(_lib.HYPIC_EUNSUPPORTED, "q/k/v must be bfloat16 or float32")


def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _host_i32(x):
    if isinstance(x, torch.Tensor):
        x = x.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _index_pair(host, dev, device, name="index array"):
    h = _host_i32(host)
    if h.ndim != 1:
        C.fail("%s must be one-dimensional" % name)
    if dev is None:
        dev = torch.from_numpy(h.copy()).to(device)
    C.device_index(name, dev, h, device)
    return h, dev


def _hptr(h):
    return h.ctypes.data_as(ctypes.c_void_p)


def _workspace(op, dims, n, device):
    lib = _lib.load()
    need = lib.hypic_workspace_bytes(op, ctypes.byref(dims), n)
    if need == 0:
        return None, 0
    key = (str(device), op)
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < need:
        buf = torch.empty(need, dtype=torch.uint8, device=device)
        _ws_cache[key] = buf
    return buf, need


def make_dims(q, v, chunk, h_qk=None):
    return Dims(h_qk=q.shape[1] if h_qk is None else h_qk, h_v=v.shape[1], d_k=q.shape[2],
                d_v=v.shape[2], dtype=_dtype_code(q), chunk=chunk)


def build_segment(q, k, v, beta, log_alpha, cu_seqlens, cu_seqlens_dev=None, *, chunk=64,
                  want_operator=True, want_o=True):
    """Zero-start build of every segment of a packed batch.

    q, k [T, h_qk, d_k], v [T, h_v, d_v] (bf16 or f32, CUDA); beta, log_alpha
    [T, h_v] float32; cu_seqlens host int32 [n_seg + 1].
    Returns dict(o, S_seg, P_hat, log_decay) of torch tensors (o / P_hat /
    log_decay are None when not requested).
    """
    lib = _lib.load()
    T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
    dev = q.device
    C.per_token("beta", beta, T, h_v, dev)
    C.per_token("log_alpha", log_alpha, T, h_v, dev)
    dims = make_dims(q, v, chunk)
    cu_h, cu_d = _index_pair(cu_seqlens, cu_seqlens_dev, dev, "cu_seqlens")
    n_seg = len(cu_h) - 1
    o = torch.empty((T, h_v, d_v), dtype=q.dtype, device=dev) if want_o else None
    S_seg = torch.empty((n_seg, h_v, d_k, d_v), dtype=torch.float32, device=dev)
    P_hat = (torch.empty((n_seg, h_v, d_k, d_k), dtype=torch.float32, device=dev)
             if want_operator else None)
    log_decay = torch.empty((n_seg, h_v), dtype=torch.float32, device=dev) if want_operator else None
    ws, ws_bytes = _workspace(_lib.HYPIC_OP_BUILD, dims, n_seg, dev)
    _lib.check(lib.hypic_build_segment(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(log_alpha), T,
        _ptr(cu_d), _hptr(cu_h), n_seg, _ptr(o), _ptr(S_seg), _ptr(P_hat), _ptr(log_decay),
        _ptr(ws), ws_bytes, _stream(dev)))
    return {"o": o, "S_seg": S_seg, "P_hat": P_hat, "log_decay": log_decay}


def compose_segments(P_hat, log_decay, S_seg, seg_ids, req_offsets, S_prefix=None, *,
                     seg_ids_dev=None, req_offsets_dev=None, precision="split",
                     want_incoming=True, h_qk=None):
    """Eq. (6) composition of pool tuples for each request (CSR lists).

    precision: "split" (three-term split-bf16 matrix cores) or "f32".
    Returns (S_out [n_req, h_v, d_k, d_v], S_incoming [nnz, h_v, d_k, d_v] or None).
    """
    lib = _lib.load()
    if precision not in ("split", "f32"):
        C.fail("precision must be 'split' or 'f32'")
    n_pool, h_v, d_k, d_v = C.pool(P_hat, log_decay, S_seg)
    dev = S_seg.device
    dims = Dims(h_qk=h_v if h_qk is None else h_qk, h_v=h_v, d_k=d_k, d_v=d_v,
                dtype=_lib.HYPIC_F32 if precision == "f32" else _lib.HYPIC_BF16, chunk=64)
    ids_h, ids_d = _index_pair(seg_ids, seg_ids_dev, dev, "seg_ids")
    off_h, off_d = _index_pair(req_offsets, req_offsets_dev, dev, "req_offsets")
    n_req = len(off_h) - 1
    if n_req < 0:
        C.fail("req_offsets needs at least one value")
    nnz = int(off_h[-1])
    if nnz != len(ids_h):
        C.fail("req_offsets[-1] = %d but seg_ids holds %d ids" % (nnz, len(ids_h)))
    C.state("S_prefix", S_prefix, n_req, h_v, d_k, d_v, dev)
    S_out = torch.empty((n_req, h_v, d_k, d_v), dtype=torch.float32, device=dev)
    S_inc = (torch.empty((nnz, h_v, d_k, d_v), dtype=torch.float32, device=dev)
             if want_incoming else None)
    _lib.check(lib.hypic_compose_segments(
        ctypes.byref(dims), _ptr(P_hat), _ptr(log_decay), _ptr(S_seg), n_pool, _ptr(ids_d),
        _hptr(ids_h), _ptr(off_d), _hptr(off_h), n_req, _ptr(S_prefix), _ptr(S_out),
        _ptr(S_inc), None, 0, _stream(dev)))
    return S_out, S_inc


def seam_rescan(q, k, v, beta, log_alpha, tok_start, tok_len, w, S_in, *, tok_start_dev=None,
                tok_len_dev=None, chunk=64, want_post=True):
    """Seam-window rescan of each entry's first min(w, tok_len) tokens from S_in.

    Returns (o_seam [n_entries, w, h_v, d_v] (rows >= w_eff left unwritten),
    S_post [n_entries, h_v, d_k, d_v] or None).
    """
    lib = _lib.load()
    T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
    dev = q.device
    C.per_token("beta", beta, T, h_v, dev)
    C.per_token("log_alpha", log_alpha, T, h_v, dev)
    dims = make_dims(q, v, chunk)
    st_h, st_d = _index_pair(tok_start, tok_start_dev, dev, "tok_start")
    ln_h, ln_d = _index_pair(tok_len, tok_len_dev, dev, "tok_len")
    n_e = len(st_h)
    if len(ln_h) != n_e:
        C.fail("tok_start and tok_len differ in length")
    C.state("S_in", S_in, n_e, h_v, d_k, d_v, dev)
    if int(w) < 1:
        C.fail("seam width must be at least 1")
    o_seam = torch.empty((n_e, w, h_v, d_v), dtype=q.dtype, device=dev)
    S_post = torch.empty((n_e, h_v, d_k, d_v), dtype=torch.float32, device=dev) if want_post else None
    _lib.check(lib.hypic_seam_rescan(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(log_alpha), T,
        _ptr(st_d), _ptr(ln_d), _hptr(st_h), _hptr(ln_h), n_e, int(w), _ptr(S_in), _ptr(o_seam),
        _ptr(S_post), None, 0, _stream(dev)))
    return o_seam, S_post


# ---------------------------------------------------------------------------
# scalar and diagonal transition families (Tab. 1, Tab. 3)
# ---------------------------------------------------------------------------

FAMILIES = {"scalar": _lib.HYPIC_FAMILY_SCALAR, "diagonal": _lib.HYPIC_FAMILY_DIAGONAL}


def _family_code(family):
    if family not in FAMILIES:
        raise HypicError(_lib.HYPIC_EUNSUPPORTED, "family must be 'scalar' or 'diagonal'")
    return FAMILIES[family]


def family_build(family, q, k, v, gate, cu_seqlens, cu_seqlens_dev=None, *, want_o=True):
    """Zero-start build of every segment of a scalar- or diagonal-family layer.

    gate: [T, h_v] (scalar) or [T, h_v, d_k] (diagonal) float32, natural-log
    units.  Returns dict(o, S_seg, log_decay); log_decay is [n_seg, h_v] or
    [n_seg, h_v, d_k].
    """
    lib = _lib.load()
    code = _family_code(family)
    T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
    dev = q.device
    C.per_token("gate", gate, T, h_v, dev, None if family == "scalar" else d_k)
    dims = make_dims(q, v, 64)
    cu_h, cu_d = _index_pair(cu_seqlens, cu_seqlens_dev, dev, "cu_seqlens")
    n_seg = len(cu_h) - 1
    o = torch.empty((T, h_v, d_v), dtype=q.dtype, device=dev) if want_o else None
    S_seg = torch.empty((n_seg, h_v, d_k, d_v), dtype=torch.float32, device=dev)
    ld_shape = (n_seg, h_v) if family == "scalar" else (n_seg, h_v, d_k)
    log_decay = torch.empty(ld_shape, dtype=torch.float32, device=dev)
    ws, ws_bytes = _workspace(_lib.HYPIC_OP_BUILD, dims, n_seg, dev)
    _lib.check(lib.hypic_family_build(
        ctypes.byref(dims), code, _ptr(q), _ptr(k), _ptr(v), _ptr(gate), T, _ptr(cu_d),
        _hptr(cu_h), n_seg, _ptr(o), _ptr(S_seg), _ptr(log_decay), _ptr(ws), ws_bytes,
        _stream(dev)))
    return {"o": o, "S_seg": S_seg, "log_decay": log_decay}


def family_compose(family, log_decay, S_seg, seg_ids, req_offsets, S_prefix=None, *,
                   seg_ids_dev=None, req_offsets_dev=None, want_incoming=True):
    """Eq. (6) with the compressed operators of Tab. 3 for each request (CSR
    lists).  Returns (S_out, S_incoming or None)."""
    lib = _lib.load()
    code = _family_code(family)
    if not isinstance(S_seg, torch.Tensor) or S_seg.dim() != 4:
        C.fail("S_seg must be a 4-d torch tensor")
    n_pool, h_v, d_k, d_v = C.pool(None, log_decay, S_seg,
                                   None if family == "scalar" else S_seg.shape[2])
    dev = S_seg.device
    dims = Dims(h_qk=h_v, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_lib.HYPIC_F32, chunk=64)
    ids_h, ids_d = _index_pair(seg_ids, seg_ids_dev, dev, "seg_ids")
    off_h, off_d = _index_pair(req_offsets, req_offsets_dev, dev, "req_offsets")
    n_req = len(off_h) - 1
    if n_req < 0:
        C.fail("req_offsets needs at least one value")
    nnz = int(off_h[-1])
    if nnz != len(ids_h):
        C.fail("req_offsets[-1] = %d but seg_ids holds %d ids" % (nnz, len(ids_h)))
    C.state("S_prefix", S_prefix, n_req, h_v, d_k, d_v, dev)
    S_out = torch.empty((n_req, h_v, d_k, d_v), dtype=torch.float32, device=dev)
    S_inc = (torch.empty((nnz, h_v, d_k, d_v), dtype=torch.float32, device=dev)
             if want_incoming else None)
    _lib.check(lib.hypic_family_compose(
        ctypes.byref(dims), code, _ptr(log_decay), _ptr(S_seg), n_pool, _ptr(ids_d),
        _hptr(ids_h), _ptr(off_d), _hptr(off_h), n_req, _ptr(S_prefix), _ptr(S_out),
        _ptr(S_inc), None, 0, _stream(dev)))
    return S_out, S_inc


def family_seam(family, q, k, v, gate, tok_start, tok_len, w, S_in, *, tok_start_dev=None,
                tok_len_dev=None, want_post=True):
    """Seam rescan of each entry's first min(w, tok_len) tokens from S_in for a
    scalar- or diagonal-family layer.  Returns (o_seam, S_post or None)."""
    lib = _lib.load()
    code = _family_code(family)
    T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
    dev = q.device
    C.per_token("gate", gate, T, h_v, dev, None if family == "scalar" else d_k)
    dims = make_dims(q, v, 64)
    st_h, st_d = _index_pair(tok_start, tok_start_dev, dev, "tok_start")
    ln_h, ln_d = _index_pair(tok_len, tok_len_dev, dev, "tok_len")
    n_e = len(st_h)
    if len(ln_h) != n_e:
        C.fail("tok_start and tok_len differ in length")
    C.state("S_in", S_in, n_e, h_v, d_k, d_v, dev)
    if int(w) < 1:
        C.fail("seam width must be at least 1")
    o_seam = torch.empty((n_e, w, h_v, d_v), dtype=q.dtype, device=dev)
    S_post = torch.empty((n_e, h_v, d_k, d_v), dtype=torch.float32, device=dev) if want_post else None
    _lib.check(lib.hypic_family_seam(
        ctypes.byref(dims), code, _ptr(q), _ptr(k), _ptr(v), _ptr(gate), T, _ptr(st_d),
        _ptr(ln_d), _hptr(st_h), _hptr(ln_h), n_e, int(w), _ptr(S_in), _ptr(o_seam),
        _ptr(S_post), None, 0, _stream(dev)))
    return o_seam, S_post


# ---------------------------------------------------------------------------
# the KDA row of Tab. 1 (delta rule with a per-channel gate)
# ---------------------------------------------------------------------------

def kda_build(q, k, v, beta, gate, cu_seqlens, cu_seqlens_dev=None, *, want_o=True,
              want_operator=True):
    """Zero-start build of every segment of a KDA layer.

    beta: [T, h_v] float32; gate: [T, h_v, d_k] float32 per-channel log gates.
    Returns dict(o, S_seg, P_hat, log_decay) with T_C = exp(log_decay) P_hat
    (P_hat and log_decay None without the operator); the tuples compose with
    compose_segments.
    """
    lib = _lib.load()
    T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
    dev = q.device
    C.per_token("beta", beta, T, h_v, dev)
    C.per_token("gate", gate, T, h_v, dev, d_k)
    dims = make_dims(q, v, 64)
    cu_h, cu_d = _index_pair(cu_seqlens, cu_seqlens_dev, dev, "cu_seqlens")
    n_seg = len(cu_h) - 1
    o = torch.empty((T, h_v, d_v), dtype=q.dtype, device=dev) if want_o else None
    S_seg = torch.empty((n_seg, h_v, d_k, d_v), dtype=torch.float32, device=dev)
    P_hat = (torch.empty((n_seg, h_v, d_k, d_k), dtype=torch.float32, device=dev)
             if want_operator else None)
    log_decay = torch.empty((n_seg, h_v), dtype=torch.float32, device=dev) if want_operator else None
    ws, ws_bytes = _workspace(_lib.HYPIC_OP_BUILD, dims, n_seg, dev)
    _lib.check(lib.hypic_kda_build(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(gate), T, _ptr(cu_d),
        _hptr(cu_h), n_seg, _ptr(o), _ptr(S_seg), _ptr(P_hat), _ptr(log_decay), _ptr(ws),
        ws_bytes, _stream(dev)))
    return {"o": o, "S_seg": S_seg, "P_hat": P_hat, "log_decay": log_decay}


def kda_seam(q, k, v, beta, gate, tok_start, tok_len, w, S_in, *, tok_start_dev=None,
             tok_len_dev=None, want_post=True):
    """Seam rescan of each entry's first min(w, tok_len) tokens from S_in for a
    KDA layer.  Returns (o_seam, S_post or None)."""
    lib = _lib.load()
    T, h_qk, h_v, d_k, d_v = C.token_arrays(q, k, v)
    dev = q.device
    C.per_token("beta", beta, T, h_v, dev)
    C.per_token("gate", gate, T, h_v, dev, d_k)
    dims = make_dims(q, v, 64)
    st_h, st_d = _index_pair(tok_start, tok_start_dev, dev, "tok_start")
    ln_h, ln_d = _index_pair(tok_len, tok_len_dev, dev, "tok_len")
    n_e = len(st_h)
    if len(ln_h) != n_e:
        C.fail("tok_start and tok_len differ in length")
    C.state("S_in", S_in, n_e, h_v, d_k, d_v, dev)
    if int(w) < 1:
        C.fail("seam width must be at least 1")
    o_seam = torch.empty((n_e, w, h_v, d_v), dtype=q.dtype, device=dev)
    S_post = torch.empty((n_e, h_v, d_k, d_v), dtype=torch.float32, device=dev) if want_post else None
    _lib.check(lib.hypic_kda_seam(
        ctypes.byref(dims), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(gate), T, _ptr(st_d),
        _ptr(ln_d), _hptr(st_h), _hptr(ln_h), n_e, int(w), _ptr(S_in), _ptr(o_seam),
        _ptr(S_post), None, 0, _stream(dev)))
    return o_seam, S_post


# ---------------------------------------------------------------------------
# reuse-time steps: RoPE state shift (Eq. (7)), key re-rotation (Eq. (8)),
# causal conv with carried state (Sec. 4.2)
# ---------------------------------------------------------------------------

def _device_i32(x, device, n, name):
    """A device int32 tensor of n values as is, else a synchronous copy of host values."""
    if isinstance(x, torch.Tensor) and x.is_cuda:
        return C.device_index(name, x, range(n), device)
    h, d = _index_pair(x, None, device, name)
    if len(h) != n:
        C.fail("%s must hold %d values, got %d" % (name, n, len(h)))
    return d


def _float_states(name, S):
    if not isinstance(S, torch.Tensor) or S.dim() != 4:
        C.fail("%s must be a 4-d torch tensor" % name)
    if not S.is_cuda:
        C.fail("%s must be on a GPU" % name)
    return C.state(name, S, *S.shape, S.device)


def rope_shift_state(S, delta, base=10000.0, out=None):
    """S [n, h_v, d_k, d_v] float32 -> R(delta[e]) S[e, h] (out may be S).
    delta: [n] int32, a device tensor or host values."""
    lib = _lib.load()
    _float_states("S", S)
    n, h_v, d_k, d_v = S.shape
    dev = S.device
    dims = Dims(h_qk=h_v, h_v=h_v, d_k=d_k, d_v=d_v, dtype=_lib.HYPIC_F32, chunk=64)
    dl = _device_i32(delta, dev, n, "delta")
    out = torch.empty_like(S) if out is None else C.state("out", out, n, h_v, d_k, d_v, dev)
    _lib.check(lib.hypic_rope_shift_state(ctypes.byref(dims), _ptr(S), _ptr(out), n, _ptr(dl),
                                          float(base), _stream(dev)))
    return out


def rope_rerotate_keys(k, cu_seqlens, delta, base=10000.0, out=None, cu_seqlens_dev=None):
    """k [T, h, d] (bf16 or f32) -> R(delta[s]) k for the tokens of segment s.
    delta: [n_seg] int32, a device tensor or host values."""
    lib = _lib.load()
    if not isinstance(k, torch.Tensor) or k.dim() != 3 or not k.is_cuda:
        C.fail("k must be a 3-d torch tensor on a GPU")
    T, h, d = k.shape
    dev = k.device
    C._tensor("k", k, k.dtype, (T, h, d), dev)
    dims = Dims(h_qk=h, h_v=h, d_k=d, d_v=d, dtype=_dtype_code(k), chunk=64)
    cu_h, cu_d = _index_pair(cu_seqlens, cu_seqlens_dev, dev, "cu_seqlens")
    if len(cu_h) < 1 or int(cu_h[-1]) > T:
        C.fail("cu_seqlens must end at or before the %d key rows" % T)
    dl = _device_i32(delta, dev, len(cu_h) - 1, "delta")
    out = torch.empty_like(k) if out is None else C._tensor("out", out, k.dtype, (T, h, d), dev)
    _lib.check(lib.hypic_rope_rerotate_keys(ctypes.byref(dims), _ptr(k), _ptr(out), _ptr(cu_d),
                                            _hptr(cu_h), len(cu_h) - 1, _ptr(dl), float(base),
                                            _stream(dev)))
    return out


def causal_conv(x, weight, cu_seqlens, state_in=None, *, silu=True, want_state=True,
                cu_seqlens_dev=None):
    """x [T, C] (bf16 or f32), weight [C, K] float32 -> (y [T, C], state_out
    [n_seg, K - 1, C] float32 or None)."""
    lib = _lib.load()
    if not isinstance(x, torch.Tensor) or x.dim() != 2 or not x.is_cuda:
        C.fail("x must be a 2-d torch tensor on a GPU")
    T, ch = x.shape
    dev = x.device
    C._tensor("x", x, x.dtype, (T, ch), dev)
    if not isinstance(weight, torch.Tensor) or weight.dim() != 2:
        C.fail("weight must be a 2-d torch tensor")
    K = weight.shape[1]
    C._tensor("weight", weight, torch.float32, (ch, K), dev)
    cu_h, cu_d = _index_pair(cu_seqlens, cu_seqlens_dev, dev, "cu_seqlens")
    n_seg = len(cu_h) - 1
    if n_seg >= 0 and int(cu_h[-1]) > T:
        C.fail("cu_seqlens must end at or before the %d input rows" % T)
    if state_in is not None:
        C._tensor("state_in", state_in, torch.float32, (n_seg, K - 1, ch), dev)
    y = torch.empty_like(x)
    st_out = (torch.empty((n_seg, K - 1, ch), dtype=torch.float32, device=dev)
              if want_state else None)
    _lib.check(lib.hypic_causal_conv(_dtype_code(x), ch, K, _ptr(x), _ptr(weight), _ptr(cu_d),
                                     _hptr(cu_h), n_seg, _ptr(state_in), _ptr(y), _ptr(st_out),
                                     1 if silu else 0, _stream(dev)))
    return y, st_out


# ---------------------------------------------------------------------------
# reuse with seam windows that advance the state (Sec. 4.3)
# ---------------------------------------------------------------------------

def compose_and_rescan(P_hat, log_decay, S_seg, q, k, v, beta, log_alpha, seam_start, seam_len,
                       w, seg_ids, req_offsets, S_prefix=None):
    """Eq. (6) composition of whole-segment pool tuples with each listed entry's
    first min(w, seam_len) tokens rescanned from the state entering it, in one
    pass (see include/hypic.h; bf16 tokens, w <= 64).
    Returns (S_out [n_req, h_v, d_k, d_v], o_seam [nnz, w, h_v, d_v])."""
    return _seam_compose("hypic_compose_and_rescan", P_hat, log_decay, S_seg, q, k, v, beta,
                         log_alpha, seam_start, seam_len, w, seg_ids, req_offsets, S_prefix)


def compose_with_seams(P_hat, log_decay, S_seg, q, k, v, beta, log_alpha, seam_start, seam_len,
                       w, seg_ids, req_offsets, S_prefix=None):
    """Tail tuples of the pool composed with each entry's seam run from the
    running state first (see include/hypic.h).  Token dtype gives the
    composition arithmetic (bf16: split bf16; f32: float32 matrix cores).
    Returns (S_out [n_req, h_v, d_k, d_v], o_seam [nnz, w, h_v, d_v])."""
    return _seam_compose("hypic_compose_with_seams", P_hat, log_decay, S_seg, q, k, v, beta,
                         log_alpha, seam_start, seam_len, w, seg_ids, req_offsets, S_prefix)


def _seam_compose(entry, P_hat, log_decay, S_seg, q, k, v, beta, log_alpha, seam_start, seam_len,
                  w, seg_ids, req_offsets, S_prefix):
    lib = _lib.load()
    n_pool, h_v, d_k, d_v = C.pool(P_hat, log_decay, S_seg)
    dev = S_seg.device
    T, h_qk, h_vt, d_kt, d_vt = C.token_arrays(q, k, v)
    if (h_vt, d_kt, d_vt) != (h_v, d_k, d_v) or q.device != dev:
        C.fail("token arrays (%d heads, %d x %d) do not match the pool (%d heads, %d x %d)"
               % (h_vt, d_kt, d_vt, h_v, d_k, d_v))
    C.per_token("beta", beta, T, h_v, dev)
    C.per_token("log_alpha", log_alpha, T, h_v, dev)
    dims = make_dims(q, v, 64)
    ss_h, ss_d = _index_pair(seam_start, None, dev, "seam_start")
    sl_h, sl_d = _index_pair(seam_len, None, dev, "seam_len")
    if len(ss_h) != n_pool or len(sl_h) != n_pool:
        C.fail("seam_start and seam_len must hold one value per pool entry (%d)" % n_pool)
    ids_h, ids_d = _index_pair(seg_ids, None, dev, "seg_ids")
    off_h, off_d = _index_pair(req_offsets, None, dev, "req_offsets")
    n_req = len(off_h) - 1
    if n_req < 0:
        C.fail("req_offsets needs at least one value")
    nnz = int(off_h[-1])
    if nnz != len(ids_h):
        C.fail("req_offsets[-1] = %d but seg_ids holds %d ids" % (nnz, len(ids_h)))
    C.state("S_prefix", S_prefix, n_req, h_v, d_k, d_v, dev)
    if int(w) < 1:
        C.fail("seam width must be at least 1")
    max_n = int(np.max(np.diff(off_h))) if n_req > 0 else 0
    S_out = torch.empty((n_req, h_v, d_k, d_v), dtype=torch.float32, device=dev)
    o_seam = torch.empty((nnz, w, h_v, d_v), dtype=q.dtype, device=dev)
    if entry == "hypic_compose_with_seams":
        need = lib.hypic_seam_compose_workspace_bytes(ctypes.byref(dims), n_req, max_n)
    else:
        need = lib.hypic_workspace_bytes(_lib.HYPIC_OP_COMPOSE_RESCAN, ctypes.byref(dims), n_req)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _lib.check(getattr(lib, entry)(
        ctypes.byref(dims), _ptr(P_hat), _ptr(log_decay), _ptr(S_seg), n_pool, _ptr(q), _ptr(k),
        _ptr(v), _ptr(beta), _ptr(log_alpha), q.shape[0], _ptr(ss_d), _hptr(ss_h), _ptr(sl_d),
        _hptr(sl_h), int(w), _ptr(ids_d), _hptr(ids_h), _ptr(off_d), _hptr(off_h), n_req,
        _ptr(S_prefix), _ptr(S_out), _ptr(o_seam), _ptr(ws), need, _stream(dev)))
    return S_out, o_seam
