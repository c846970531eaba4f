"""Host-side tensor checks in front of the C ABI (CPU only): a bf16 beta, a
float32 v next to a bf16 q, a short P_hat or a short incoming state is
rejected with HypicError(HYPIC_EINVAL) before anything is launched.  The GPU
requirement is switched off so the shape and dtype logic runs on CPU tensors."""

import pytest
import torch

from paper_2607_01299_amd import _checks as C
from paper_2607_01299_amd import _lib

cpu = torch.device("cpu")


def _tok(T=10, h_qk=2, h_v=4, d_k=64, d_v=128, dt=torch.bfloat16):
    return (torch.zeros(T, h_qk, d_k, dtype=dt), torch.zeros(T, h_qk, d_k, dtype=dt),
            torch.zeros(T, h_v, d_v, dtype=dt))


def _rejects(fn, *a, **kw):
    with pytest.raises(_lib.HypicError) as e:
        fn(*a, **kw)
    assert e.value.code == _lib.HYPIC_EINVAL
    return str(e.value)


def test_token_arrays_accept_matching_tensors():
    assert C.token_arrays(*_tok(), require_gpu=False) == (10, 2, 4, 64, 128)


def test_token_arrays_reject_mismatches():
    q, k, v = _tok()
    assert "v must be" in _rejects(C.token_arrays, q, k, v.float(), require_gpu=False)
    assert "k must have shape" in _rejects(C.token_arrays, q, k[:9], v, require_gpu=False)
    assert "token rows" in _rejects(C.token_arrays, q, k, v[:9], require_gpu=False)
    assert "multiple" in _rejects(C.token_arrays, *_tok(h_qk=3, h_v=4), require_gpu=False)
    assert "bfloat16 or float32" in _rejects(C.token_arrays, q.half(), k.half(), v.half(),
                                             require_gpu=False)
    qt = torch.zeros(64, 2, 10, dtype=torch.bfloat16).permute(2, 1, 0)
    assert "contiguous" in _rejects(C.token_arrays, qt, qt.contiguous(),
                                    torch.zeros(10, 2, 64, dtype=torch.bfloat16),
                                    require_gpu=False)
    assert "on a GPU" in _rejects(C.token_arrays, q, k, v)


def test_per_token_and_state_shapes():
    C.per_token("beta", torch.zeros(10, 4), 10, 4, cpu)
    assert "float32" in _rejects(C.per_token, "beta", torch.zeros(10, 4, dtype=torch.bfloat16),
                                 10, 4, cpu)
    assert "shape" in _rejects(C.per_token, "gate", torch.zeros(10, 4), 10, 4, cpu, 64)
    assert C.state("S_in", None, 3, 4, 64, 64, cpu) is None
    assert "shape" in _rejects(C.state, "S_in", torch.zeros(2, 4, 64, 64), 3, 4, 64, 64, cpu)


def test_pool_rejects_short_or_mistyped_parts():
    S = torch.zeros(8, 4, 64, 128)
    P = torch.zeros(8, 4, 64, 64)
    g = torch.zeros(8, 4)
    assert C.pool(P, g, S, require_gpu=False) == (8, 4, 64, 128)
    assert "P_hat" in _rejects(C.pool, P[:7], g, S, require_gpu=False)
    assert "log_decay" in _rejects(C.pool, P, g[:7], S, require_gpu=False)
    assert "log_decay" in _rejects(C.pool, None, g, S, 64, require_gpu=False)
    assert "P_hat" in _rejects(C.pool, P.double(), g, S, require_gpu=False)


def test_device_index_length_and_type():
    C.device_index("cu", torch.zeros(3, dtype=torch.int32), [0, 1, 2], cpu)
    assert "holds" in _rejects(C.device_index, "cu", torch.zeros(2, dtype=torch.int32),
                               [0, 1, 2], cpu)
    assert "int32" in _rejects(C.device_index, "cu", torch.zeros(3, dtype=torch.int64),
                               [0, 1, 2], cpu)
