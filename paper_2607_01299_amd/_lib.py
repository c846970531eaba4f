"""ctypes binding of libhypic.so (declarations in include/hypic.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels.  If the library has not been built, every call raises -- there is no
fallback path.
"""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhypic.so")

HYPIC_OK = 0
HYPIC_EINVAL = -1
HYPIC_EUNSUPPORTED = -2
HYPIC_EWORKSPACE = -3
HYPIC_EHIP = -4

HYPIC_F32 = 0
HYPIC_BF16 = 1

HYPIC_OP_BUILD = 0
HYPIC_OP_COMPOSE = 1
HYPIC_OP_SEAM = 2
HYPIC_OP_COMPOSE_RESCAN = 3

EXPORTS = (
    "hypic_workspace_bytes",
    "hypic_status_str",
    "hypic_build_segment",
    "hypic_compose_segments",
    "hypic_seam_rescan",
    "hypic_family_build",
    "hypic_family_compose",
    "hypic_family_seam",
    "hypic_rope_shift_state",
    "hypic_rope_rerotate_keys",
    "hypic_causal_conv",
    "hypic_seam_compose_workspace_bytes",
    "hypic_compose_with_seams",
    "hypic_kda_build",
    "hypic_kda_seam",
    "hypic_build_segment_noalloc",
    "hypic_compose_and_rescan",
)

HYPIC_NOALLOC_MAX_SEGMENTS = 65536

HYPIC_FAMILY_SCALAR = 1
HYPIC_FAMILY_DIAGONAL = 2


class HypicError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("hypic error %d: %s" % (code, msg))
        self.code = code


class Dims(ctypes.Structure):
    _fields_ = [
        ("h_qk", ctypes.c_int32),
        ("h_v", ctypes.c_int32),
        ("d_k", ctypes.c_int32),
        ("d_v", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("chunk", ctypes.c_int32),
    ]


_lib = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t


def load():
    """Load libhypic.so once; raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise HypicError(HYPIC_EHIP, "libhypic.so not built at %s (run "
                         "`python -m paper_2607_01299_amd.build`)" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    lib.hypic_workspace_bytes.argtypes = [_I32, ctypes.POINTER(Dims), ctypes.c_int64]
    lib.hypic_workspace_bytes.restype = _SZ
    lib.hypic_status_str.argtypes = [_I32]
    lib.hypic_status_str.restype = ctypes.c_char_p
    lib.hypic_build_segment.argtypes = [
        ctypes.POINTER(Dims), _P, _P, _P, _P, _P, _I32, _P, _P, _I32, _P, _P, _P, _P, _P, _SZ,
        _P]
    lib.hypic_build_segment.restype = _I32
    lib.hypic_build_segment_noalloc.argtypes = [
        ctypes.POINTER(Dims), _P, _P, _P, _P, _P, _I32, _P, _P, _I32, _P, _P, _P, _P, _P]
    lib.hypic_build_segment_noalloc.restype = _I32
    lib.hypic_compose_segments.argtypes = [
        ctypes.POINTER(Dims), _P, _P, _P, _I32, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _SZ, _P]
    lib.hypic_compose_segments.restype = _I32
    lib.hypic_seam_rescan.argtypes = [
        ctypes.POINTER(Dims), _P, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _I32, _I32, _P, _P, _P,
        _P, _SZ, _P]
    lib.hypic_seam_rescan.restype = _I32
    lib.hypic_family_build.argtypes = [
        ctypes.POINTER(Dims), _I32, _P, _P, _P, _P, _I32, _P, _P, _I32, _P, _P, _P, _P, _SZ, _P]
    lib.hypic_family_build.restype = _I32
    lib.hypic_family_compose.argtypes = [
        ctypes.POINTER(Dims), _I32, _P, _P, _I32, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _SZ, _P]
    lib.hypic_family_compose.restype = _I32
    lib.hypic_family_seam.argtypes = [
        ctypes.POINTER(Dims), _I32, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _I32, _I32, _P, _P, _P,
        _P, _SZ, _P]
    lib.hypic_family_seam.restype = _I32
    lib.hypic_rope_shift_state.argtypes = [ctypes.POINTER(Dims), _P, _P, _I32, _P, ctypes.c_double,
                                           _P]
    lib.hypic_rope_shift_state.restype = _I32
    lib.hypic_rope_rerotate_keys.argtypes = [ctypes.POINTER(Dims), _P, _P, _P, _P, _I32, _P,
                                             ctypes.c_double, _P]
    lib.hypic_rope_rerotate_keys.restype = _I32
    lib.hypic_causal_conv.argtypes = [_I32, _I32, _I32, _P, _P, _P, _P, _I32, _P, _P, _P, _I32, _P]
    lib.hypic_causal_conv.restype = _I32
    lib.hypic_kda_build.argtypes = [
        ctypes.POINTER(Dims), _P, _P, _P, _P, _P, _I32, _P, _P, _I32, _P, _P, _P, _P, _P, _SZ,
        _P]
    lib.hypic_kda_build.restype = _I32
    lib.hypic_kda_seam.argtypes = [
        ctypes.POINTER(Dims), _P, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _I32, _I32, _P, _P, _P,
        _P, _SZ, _P]
    lib.hypic_kda_seam.restype = _I32
    lib.hypic_seam_compose_workspace_bytes.argtypes = [ctypes.POINTER(Dims), _I32, _I32]
    lib.hypic_seam_compose_workspace_bytes.restype = _SZ
    lib.hypic_compose_with_seams.argtypes = [
        ctypes.POINTER(Dims), _P, _P, _P, _I32, _P, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _I32,
        _P, _P, _P, _P, _I32, _P, _P, _P, _P, _SZ, _P]
    lib.hypic_compose_with_seams.restype = _I32
    lib.hypic_compose_and_rescan.argtypes = lib.hypic_compose_with_seams.argtypes
    lib.hypic_compose_and_rescan.restype = _I32
    _lib = lib
    return lib


def check(code):
    if code != HYPIC_OK:
        raise HypicError(code, load().hypic_status_str(code).decode())
