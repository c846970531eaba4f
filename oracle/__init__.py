"""Float64 CPU oracle for the gated-delta-rule segment cache (Hypic).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.  The
product path (the HIP library and its Python binding) never imports, calls or
links it, and this package never imports the product path.
"""

from .gdn import (  # noqa: F401
    qk_head_of,
    recurrence,
    segment_operator,
    build_segments,
    compose,
    seam,
    compose_with_seams,
)
from . import families  # noqa: F401,E402  (scalar / diagonal families, RoPE, conv)
from . import kda  # noqa: F401,E402  (the KDA row of Tab. 1)
