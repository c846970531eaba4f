"""Host-side checks of the torch tensors handed to the C ABI.

The C ABI validates sizes, offsets and alignment, but it sees only pointers:
it cannot tell a float32 beta from a bf16 one, or a short P_hat from a full
one.  These checks compare dtype, shape, device and layout of every tensor
with what include/hypic.h specifies for it, before anything is launched, and
raise HypicError(HYPIC_EINVAL) naming the argument.
"""

import torch

from . import _lib
from ._lib import HypicError

TOKEN_DTYPES = (torch.bfloat16, torch.float32)


def fail(msg):
    raise HypicError(_lib.HYPIC_EINVAL, msg)


def _tensor(name, t, dtype, shape, device):
    if not isinstance(t, torch.Tensor):
        fail("%s must be a torch tensor" % name)
    if t.dtype != dtype:
        fail("%s must be %s, got %s" % (name, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape):
        fail("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if t.device != device:
        fail("%s is on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        fail("%s must be contiguous" % name)
    return t


def token_arrays(q, k, v, require_gpu=True):
    """q, k [T, h_qk, d_k] and v [T, h_v, d_v] of one token dtype on one GPU.
    Returns (T, h_qk, h_v, d_k, d_v).  (require_gpu=False lets the host tests
    exercise the shape and dtype checks on CPU tensors.)"""
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not isinstance(t, torch.Tensor) or t.dim() != 3:
            fail("%s must be a 3-d torch tensor" % name)
    if q.dtype not in TOKEN_DTYPES:
        fail("q must be bfloat16 or float32, got %s" % q.dtype)
    if require_gpu and not q.is_cuda:
        fail("q must be on a GPU")
    T, h_qk, d_k = q.shape
    _tensor("q", q, q.dtype, (T, h_qk, d_k), q.device)
    _tensor("k", k, q.dtype, (T, h_qk, d_k), q.device)
    if v.shape[0] != T:
        fail("v must have %d token rows, got %d" % (T, v.shape[0]))
    h_v, d_v = v.shape[1], v.shape[2]
    _tensor("v", v, q.dtype, (T, h_v, d_v), q.device)
    if h_v % h_qk != 0:
        fail("v heads (%d) must be a multiple of q/k heads (%d)" % (h_v, h_qk))
    return T, h_qk, h_v, d_k, d_v


def per_token(name, t, T, h_v, device, width=None):
    """A float32 [T, h_v] (or [T, h_v, width]) array such as beta, log_alpha or a gate."""
    shape = (T, h_v) if width is None else (T, h_v, width)
    return _tensor(name, t, torch.float32, shape, device)


def state(name, t, n, h_v, d_k, d_v, device):
    """A float32 [n, h_v, d_k, d_v] array of states (None passes)."""
    if t is None:
        return None
    return _tensor(name, t, torch.float32, (n, h_v, d_k, d_v), device)


def pool(P_hat, log_decay, S_seg, ld_width=None, require_gpu=True):
    """Pool of cached tuples: S_seg [n_pool, h_v, d_k, d_v], P_hat [n_pool, h_v,
    d_k, d_k] (None for the families) and log_decay [n_pool, h_v] (or [n_pool,
    h_v, ld_width]), float32 on one GPU.  Returns (n_pool, h_v, d_k, d_v)."""
    if not isinstance(S_seg, torch.Tensor) or S_seg.dim() != 4:
        fail("S_seg must be a 4-d torch tensor")
    if require_gpu and not S_seg.is_cuda:
        fail("S_seg must be on a GPU")
    n_pool, h_v, d_k, d_v = S_seg.shape
    dev = S_seg.device
    _tensor("S_seg", S_seg, torch.float32, (n_pool, h_v, d_k, d_v), dev)
    if P_hat is not None:
        _tensor("P_hat", P_hat, torch.float32, (n_pool, h_v, d_k, d_k), dev)
    ld_shape = (n_pool, h_v) if ld_width is None else (n_pool, h_v, ld_width)
    _tensor("log_decay", log_decay, torch.float32, ld_shape, dev)
    return n_pool, h_v, d_k, d_v


def device_index(name, dev_arr, host_arr, device):
    """A device int32 copy of a host index array: same length, contiguous, on the
    inputs' GPU (its values are the caller's promise; the C ABI checks the host copy)."""
    if not isinstance(dev_arr, torch.Tensor):
        fail("%s must be a torch tensor" % name)
    if dev_arr.dtype != torch.int32 or not dev_arr.is_contiguous() or dev_arr.dim() != 1:
        fail("device index array %s must be a contiguous 1-d int32 tensor" % name)
    if dev_arr.device != device:
        fail("%s is on %s, expected %s" % (name, dev_arr.device, device))
    if dev_arr.numel() != len(host_arr):
        fail("%s holds %d values, its host copy %d" % (name, dev_arr.numel(), len(host_arr)))
    return dev_arr
