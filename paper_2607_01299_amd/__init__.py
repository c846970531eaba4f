"""MI355X (gfx950) hot path of Hypic position-independent caching for
gated-delta-rule linear-attention layers: segment build, Eq. (6) composition
and seam rescan, as HIP kernels behind the C ABI of include/hypic.h.
"""

from ._lib import HypicError  # noqa: F401


def __getattr__(name):
    # the torch-facing calls load torch lazily so that the generators and the
    # library loader stay importable without it
    if name in ("build_segment", "compose_segments", "seam_rescan", "make_dims",
                "family_build", "family_compose", "family_seam", "rope_shift_state",
                "rope_rerotate_keys", "causal_conv", "compose_with_seams", "compose_and_rescan", "kda_build",
                "kda_seam"):
        from . import ops
        return getattr(ops, name)
    raise AttributeError(name)
