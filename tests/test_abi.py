"""C ABI: the library loads, exports every declared symbol, and rejects bad
arguments on the host before touching the GPU.  CPU only: every call here
returns from validation, so nothing is launched (fake device pointers are
never dereferenced)."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2607_01299_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hypic.h")

FAKE = ctypes.c_void_p(0x10000)      # 16-byte aligned, never dereferenced
FAKE_ODD = ctypes.c_void_p(0x10004)  # misaligned


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(hypic_[a-z_]+)\s*\(", text)))


def _dims(h_qk=2, h_v=4, d_k=128, d_v=128, dtype=_lib.HYPIC_BF16, chunk=64):
    return _lib.Dims(h_qk=h_qk, h_v=h_v, d_k=d_k, d_v=d_v, dtype=dtype, chunk=chunk)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libhypic.so is not built; run `python -m paper_2607_01299_amd.build`")
    return _lib.load()


def test_every_declared_symbol_is_exported(lib):
    declared = _declared()
    assert set(declared) == set(_lib.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (hypic_\w+)", out))
    for name in declared:
        assert name in exported, name
        assert hasattr(lib, name)


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4):
        assert lib.hypic_status_str(code)
    assert lib.hypic_status_str(-99) == b"unknown status"


def test_workspace_sizes(lib):
    d = _dims()
    assert lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(d), 1000) >= 1000 * 4
    # up to 128 segments carry their order in the kernel arguments
    assert lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(d), 128) == 0
    assert lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(d), 0) == 0
    assert lib.hypic_workspace_bytes(_lib.HYPIC_OP_COMPOSE, ctypes.byref(d), 10) == 0
    bad = _dims(d_k=96)
    assert lib.hypic_workspace_bytes(_lib.HYPIC_OP_BUILD, ctypes.byref(bad), 64) == 0


def _build(lib, dims, cu, n_seg=None, q=FAKE, S=FAKE, ws=FAKE, ws_bytes=1 << 20, o=FAKE,
           cu_dev=FAKE, n_tokens=None):
    cu = np.asarray(cu, dtype=np.int32)
    n_seg = len(cu) - 1 if n_seg is None else n_seg
    n_tokens = int(cu[-1]) if n_tokens is None else n_tokens
    return lib.hypic_build_segment(
        ctypes.byref(dims) if dims is not None else None, q, FAKE, FAKE, FAKE, FAKE, n_tokens,
        cu_dev, cu.ctypes.data_as(ctypes.c_void_p), n_seg, o, S, FAKE, FAKE, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(d_k=96), _lib.HYPIC_EUNSUPPORTED),
    (dict(d_v=32), _lib.HYPIC_EUNSUPPORTED),
    (dict(chunk=48), _lib.HYPIC_EUNSUPPORTED),
    (dict(dtype=7), _lib.HYPIC_EUNSUPPORTED),
    (dict(h_qk=3, h_v=4), _lib.HYPIC_EINVAL),
    (dict(h_v=0), _lib.HYPIC_EINVAL),
])
def test_build_rejects_bad_dims(lib, kw, code):
    assert _build(lib, _dims(**kw), [0, 10, 20]) == code


def test_build_rejects_bad_arguments(lib):
    d = _dims()
    assert _build(lib, None, [0, 10]) == _lib.HYPIC_EINVAL
    assert _build(lib, d, [0, 10], q=None) == _lib.HYPIC_EINVAL
    assert _build(lib, d, [0, 10], S=None) == _lib.HYPIC_EINVAL
    assert _build(lib, d, [0, 10], cu_dev=None) == _lib.HYPIC_EINVAL
    assert _build(lib, d, [0, 10], q=FAKE_ODD) == _lib.HYPIC_EINVAL
    assert _build(lib, d, [0, 10], o=FAKE_ODD) == _lib.HYPIC_EINVAL
    assert _build(lib, d, [1, 10]) == _lib.HYPIC_EINVAL            # must start at 0
    assert _build(lib, d, [0, 10, 5]) == _lib.HYPIC_EINVAL         # decreasing
    assert _build(lib, d, [0, 10], n_seg=-1) == _lib.HYPIC_EINVAL
    # past 128 segments the order needs device workspace
    many = np.arange(0, 10 * 130, 10)
    assert _build(lib, d, many, ws=None) == _lib.HYPIC_EWORKSPACE
    assert _build(lib, d, many, ws_bytes=4) == _lib.HYPIC_EWORKSPACE
    # nothing to do is not an error (and launches nothing)
    assert _build(lib, d, [0], n_seg=0) == _lib.HYPIC_OK


def test_noalloc_build_rejects_more_segments_than_its_scratch(lib):
    """The no-allocation build holds at most HYPIC_NOALLOC_MAX_SEGMENTS orders;
    beyond that it returns HYPIC_EWORKSPACE before touching the GPU."""
    d = _dims()
    n = _lib.HYPIC_NOALLOC_MAX_SEGMENTS + 1
    cu = np.arange(n + 1, dtype=np.int32)
    code = lib.hypic_build_segment_noalloc(
        ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, n, FAKE,
        cu.ctypes.data_as(ctypes.c_void_p), n, FAKE, FAKE, FAKE, FAKE, None)
    assert code == _lib.HYPIC_EWORKSPACE
    assert "HYPIC_NOALLOC_MAX_SEGMENTS 65536" in open(HEADER).read()


def test_build_rejects_offsets_past_the_token_arrays(lib):
    """The segments must lie inside the n_tokens rows of q, k, v (and o): an
    offset past them is rejected on the host, before any launch."""
    d = _dims()
    assert _build(lib, d, [0, 10, 21], n_tokens=20) == _lib.HYPIC_EINVAL
    assert _build(lib, d, [0, 10], n_tokens=-1) == _lib.HYPIC_EINVAL
    assert _fbuild(lib, _lib.HYPIC_FAMILY_SCALAR, [0, 10, 21], n_tokens=20) == _lib.HYPIC_EINVAL
    assert _kbuild(lib, [0, 10, 21], n_tokens=20) == _lib.HYPIC_EINVAL


def _compose(lib, dims, ids, offs, n_pool=8, S_out=FAKE, P=FAKE, S_seg=FAKE, S_prefix=None,
             S_inc=None):
    ids = np.asarray(ids, dtype=np.int32)
    offs = np.asarray(offs, dtype=np.int32)
    return lib.hypic_compose_segments(
        ctypes.byref(dims), P, FAKE, S_seg, n_pool, FAKE, ids.ctypes.data_as(ctypes.c_void_p),
        FAKE, offs.ctypes.data_as(ctypes.c_void_p), len(offs) - 1, S_prefix, S_out, S_inc, None,
        0, None)


def test_compose_rejects_bad_arguments(lib):
    d = _dims()
    assert _compose(lib, d, [0, 8], [0, 2]) == _lib.HYPIC_EINVAL       # id == n_pool
    assert _compose(lib, d, [0, -1], [0, 2]) == _lib.HYPIC_EINVAL      # negative id
    assert _compose(lib, d, [0, 1], [0, 2, 1]) == _lib.HYPIC_EINVAL    # decreasing offsets
    assert _compose(lib, d, [0, 1], [1, 2]) == _lib.HYPIC_EINVAL       # must start at 0
    assert _compose(lib, d, [0, 1], [0, 2], S_out=None) == _lib.HYPIC_EINVAL
    assert _compose(lib, d, [0, 1], [0, 2], P=None) == _lib.HYPIC_EINVAL
    assert _compose(lib, _dims(d_k=32), [0], [0, 1]) == _lib.HYPIC_EUNSUPPORTED
    assert _compose(lib, d, [], [0]) == _lib.HYPIC_OK                  # no request
    # the kernel reads and writes 16-byte pieces of every state and operator
    for kw in (dict(P=FAKE_ODD), dict(S_seg=FAKE_ODD), dict(S_out=FAKE_ODD),
               dict(S_prefix=FAKE_ODD), dict(S_inc=FAKE_ODD)):
        assert _compose(lib, d, [0, 1], [0, 2], **kw) == _lib.HYPIC_EINVAL, kw


def _seam(lib, dims, start, length, w=8, n_tokens=100, o=FAKE, S_in=FAKE):
    st = np.asarray(start, dtype=np.int32)
    ln = np.asarray(length, dtype=np.int32)
    return lib.hypic_seam_rescan(
        ctypes.byref(dims), FAKE, FAKE, FAKE, FAKE, FAKE, n_tokens, FAKE, FAKE,
        st.ctypes.data_as(ctypes.c_void_p), ln.ctypes.data_as(ctypes.c_void_p), len(st), w,
        S_in, o, None, None, 0, None)


def test_seam_rejects_bad_arguments(lib):
    d = _dims()
    assert _seam(lib, d, [0, 95], [10, 10]) == _lib.HYPIC_EINVAL       # 95 + 8 > 100
    assert _seam(lib, d, [0], [0]) == _lib.HYPIC_EINVAL                # empty entry
    assert _seam(lib, d, [-1], [4]) == _lib.HYPIC_EINVAL
    assert _seam(lib, d, [0], [4], w=0) == _lib.HYPIC_EINVAL
    assert _seam(lib, d, [0], [4], o=None) == _lib.HYPIC_EINVAL
    assert _seam(lib, d, [0], [4], o=FAKE_ODD) == _lib.HYPIC_EINVAL
    assert _seam(lib, d, [0], [4], S_in=None) == _lib.HYPIC_EINVAL
    assert _seam(lib, d, [], []) == _lib.HYPIC_OK


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(_lib.HypicError):
        _lib.load()


def _fbuild(lib, family, cu, gate=FAKE, dims=None, n_tokens=None):
    cu = np.asarray(cu, dtype=np.int32)
    d = _dims() if dims is None else dims
    n_tokens = int(cu[-1]) if n_tokens is None else n_tokens
    return lib.hypic_family_build(
        ctypes.byref(d), family, FAKE, FAKE, FAKE, gate, n_tokens, FAKE,
        cu.ctypes.data_as(ctypes.c_void_p), len(cu) - 1, FAKE, FAKE, FAKE, FAKE, 1 << 20, None)


def _fcompose(lib, family, ids, offs, n_pool=8, S_out=FAKE, S_seg=FAKE):
    ids = np.asarray(ids, dtype=np.int32)
    offs = np.asarray(offs, dtype=np.int32)
    return lib.hypic_family_compose(
        ctypes.byref(_dims()), family, FAKE, S_seg, n_pool, FAKE,
        ids.ctypes.data_as(ctypes.c_void_p), FAKE, offs.ctypes.data_as(ctypes.c_void_p),
        len(offs) - 1, None, S_out, None, None, 0, None)


def _fseam(lib, family, start, length, w=8, n_tokens=100, gate=FAKE):
    st = np.asarray(start, dtype=np.int32)
    ln = np.asarray(length, dtype=np.int32)
    return lib.hypic_family_seam(
        ctypes.byref(_dims()), family, FAKE, FAKE, FAKE, gate, n_tokens, FAKE, FAKE,
        st.ctypes.data_as(ctypes.c_void_p), ln.ctypes.data_as(ctypes.c_void_p), len(st), w,
        FAKE, FAKE, None, None, 0, None)


@pytest.mark.parametrize("family", [_lib.HYPIC_FAMILY_SCALAR, _lib.HYPIC_FAMILY_DIAGONAL])
def test_family_calls_reject_bad_arguments(lib, family):
    assert _fbuild(lib, family, [0, 10, 5]) == _lib.HYPIC_EINVAL
    assert _fbuild(lib, family, [0, 10], gate=None) == _lib.HYPIC_EINVAL
    assert _fbuild(lib, family, [0, 10], dims=_dims(d_k=96)) == _lib.HYPIC_EUNSUPPORTED
    assert _fbuild(lib, family, [0]) == _lib.HYPIC_OK
    assert _fcompose(lib, family, [0, 8], [0, 2]) == _lib.HYPIC_EINVAL
    assert _fcompose(lib, family, [0, 1], [0, 2], S_out=FAKE_ODD) == _lib.HYPIC_EINVAL
    assert _fcompose(lib, family, [0, 1], [0, 2], S_seg=None) == _lib.HYPIC_EINVAL
    assert _fcompose(lib, family, [], [0]) == _lib.HYPIC_OK
    assert _fseam(lib, family, [0, 95], [10, 10]) == _lib.HYPIC_EINVAL
    assert _fseam(lib, family, [0], [4], gate=None) == _lib.HYPIC_EINVAL
    assert _fseam(lib, family, [], []) == _lib.HYPIC_OK


@pytest.mark.parametrize("family", [0, 3, -1])
def test_family_calls_reject_unknown_family(lib, family):
    assert _fbuild(lib, family, [0, 10]) == _lib.HYPIC_EUNSUPPORTED
    assert _fcompose(lib, family, [0], [0, 1]) == _lib.HYPIC_EUNSUPPORTED
    assert _fseam(lib, family, [0], [4]) == _lib.HYPIC_EUNSUPPORTED


def _kbuild(lib, cu, beta=FAKE, gate=FAKE, P_hat=FAKE, log_decay=FAKE, q=FAKE, dims=None,
            ws_bytes=1 << 20, n_tokens=None):
    cu = np.asarray(cu, dtype=np.int32)
    d = _dims() if dims is None else dims
    n_tokens = int(cu[-1]) if n_tokens is None else n_tokens
    return lib.hypic_kda_build(
        ctypes.byref(d), q, FAKE, FAKE, beta, gate, n_tokens, FAKE,
        cu.ctypes.data_as(ctypes.c_void_p), len(cu) - 1, FAKE, FAKE, P_hat, log_decay, FAKE,
        ws_bytes, None)


def _kseam(lib, start, length, w=8, n_tokens=100, gate=FAKE, S_in=FAKE):
    st = np.asarray(start, dtype=np.int32)
    ln = np.asarray(length, dtype=np.int32)
    return lib.hypic_kda_seam(
        ctypes.byref(_dims()), FAKE, FAKE, FAKE, FAKE, gate, n_tokens, FAKE, FAKE,
        st.ctypes.data_as(ctypes.c_void_p), ln.ctypes.data_as(ctypes.c_void_p), len(st), w,
        S_in, FAKE, None, None, 0, None)


def test_kda_calls_reject_bad_arguments(lib):
    assert _kbuild(lib, [0, 10, 5]) == _lib.HYPIC_EINVAL           # decreasing offsets
    assert _kbuild(lib, [3, 10]) == _lib.HYPIC_EINVAL              # offsets not from 0
    assert _kbuild(lib, [0, 10], gate=None) == _lib.HYPIC_EINVAL
    assert _kbuild(lib, [0, 10], beta=None) == _lib.HYPIC_EINVAL
    assert _kbuild(lib, [0, 10], log_decay=None) == _lib.HYPIC_EINVAL  # P_hat without log_decay
    assert _kbuild(lib, [0, 10], q=FAKE_ODD) == _lib.HYPIC_EINVAL
    assert _kbuild(lib, [0, 10], dims=_dims(d_k=96)) == _lib.HYPIC_EUNSUPPORTED
    assert _kbuild(lib, [0, 10], dims=_dims(h_qk=3, h_v=4)) != _lib.HYPIC_OK
    assert _kbuild(lib, list(range(0, 2000, 10)), ws_bytes=0) == _lib.HYPIC_EWORKSPACE
    assert _kbuild(lib, [0]) == _lib.HYPIC_OK
    assert _kseam(lib, [0, 95], [10, 10]) == _lib.HYPIC_EINVAL     # window past the tokens
    assert _kseam(lib, [0], [0]) == _lib.HYPIC_EINVAL              # empty segment
    assert _kseam(lib, [0], [4], w=0) == _lib.HYPIC_EINVAL
    assert _kseam(lib, [0], [4], gate=None) == _lib.HYPIC_EINVAL
    assert _kseam(lib, [0], [4], S_in=None) == _lib.HYPIC_EINVAL
    assert _kseam(lib, [], []) == _lib.HYPIC_OK


def test_adjacent_calls_reject_bad_arguments(lib):
    d = _dims()
    dl = FAKE
    assert lib.hypic_rope_shift_state(ctypes.byref(d), FAKE, FAKE, 3, dl, -1.0, None) == \
        _lib.HYPIC_EINVAL
    assert lib.hypic_rope_shift_state(ctypes.byref(d), FAKE_ODD, FAKE, 3, dl, 1e4, None) == \
        _lib.HYPIC_EINVAL
    assert lib.hypic_rope_shift_state(ctypes.byref(d), FAKE, FAKE, 0, dl, 1e4, None) == _lib.HYPIC_OK
    assert lib.hypic_rope_shift_state(ctypes.byref(_dims(d_k=48)), FAKE, FAKE, 3, dl, 1e4,
                                      None) == _lib.HYPIC_EUNSUPPORTED
    cu = np.array([0, 5, 3], dtype=np.int32)
    hcu = cu.ctypes.data_as(ctypes.c_void_p)
    assert lib.hypic_rope_rerotate_keys(ctypes.byref(d), FAKE, FAKE, FAKE, hcu, 2, dl, 1e4,
                                        None) == _lib.HYPIC_EINVAL
    assert lib.hypic_rope_rerotate_keys(ctypes.byref(d), FAKE, FAKE, FAKE, hcu, 1, dl,
                                        float("nan"), None) == _lib.HYPIC_EINVAL
    assert lib.hypic_causal_conv(_lib.HYPIC_BF16, 16, 9, FAKE, FAKE, FAKE, hcu, 1, None, FAKE_ODD,
                                 None, 1, None) == _lib.HYPIC_EUNSUPPORTED
    assert lib.hypic_causal_conv(_lib.HYPIC_BF16, 16, 4, FAKE, FAKE, FAKE, hcu, 2, None, FAKE_ODD,
                                 None, 1, None) == _lib.HYPIC_EINVAL     # decreasing offsets
    assert lib.hypic_causal_conv(_lib.HYPIC_BF16, 16, 4, FAKE, FAKE, FAKE, hcu, 1, None, FAKE,
                                 None, 1, None) == _lib.HYPIC_EINVAL     # y aliases x
    assert lib.hypic_causal_conv(7, 16, 4, FAKE, FAKE, FAKE, hcu, 1, None, FAKE_ODD, None, 1,
                                 None) == _lib.HYPIC_EUNSUPPORTED
    assert lib.hypic_causal_conv(_lib.HYPIC_F32, 16, 4, FAKE, FAKE, FAKE, hcu, 0, None, FAKE_ODD,
                                 None, 1, None) == _lib.HYPIC_OK


def test_compose_with_seams_rejects_bad_arguments(lib):
    d = _dims()
    ids = np.array([0, 1], dtype=np.int32)
    offs = np.array([0, 2], dtype=np.int32)
    ss = np.array([0, 10], dtype=np.int32)
    sl = np.array([10, 10], dtype=np.int32)
    h = lambda a: a.ctypes.data_as(ctypes.c_void_p)  # noqa: E731

    def call(ids=ids, offs=offs, ss=ss, sl=sl, n_pool=2, n_tokens=20, w=8, ws=FAKE, ws_bytes=1 << 30,
             o=FAKE):
        return lib.hypic_compose_with_seams(
            ctypes.byref(d), FAKE, FAKE, FAKE, n_pool, FAKE, FAKE, FAKE, FAKE, FAKE, n_tokens, FAKE,
            h(ss), FAKE, h(sl), w, FAKE, h(ids), FAKE, h(offs), len(offs) - 1, None, FAKE, o, ws,
            ws_bytes, None)

    assert call(ids=np.array([0, 2], dtype=np.int32)) == _lib.HYPIC_EINVAL      # id >= n_pool
    assert call(n_tokens=15) == _lib.HYPIC_EINVAL                                # seam past the end
    assert call(sl=np.array([10, 0], dtype=np.int32)) == _lib.HYPIC_EINVAL       # empty entry
    assert call(w=0) == _lib.HYPIC_EINVAL
    assert call(o=FAKE_ODD) == _lib.HYPIC_EINVAL
    assert call(ws=None) == _lib.HYPIC_EWORKSPACE
    need = lib.hypic_seam_compose_workspace_bytes(ctypes.byref(d), 1, 2)
    assert need >= 2 * 4 * 128 * 128 * 4
    assert call(ws_bytes=need - 1) == _lib.HYPIC_EWORKSPACE
    assert call(offs=np.array([0], dtype=np.int32)) == _lib.HYPIC_OK             # no request
