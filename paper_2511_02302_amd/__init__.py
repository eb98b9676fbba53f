"""FP8-Flow-MoE expert layer for AMD Instinct MI355X (gfx950).

libff8.so (hand-written HIP kernels behind a C ABI, declared in include/ff8.h) does
all the work; ``ff8`` is its ctypes binding (same names as the C entry points) and
``layer.ExpertLayerFP8`` strings the calls into the expert layer's forward and
backward.  Build the library with ``python -m paper_2511_02302_amd.build``.
"""

from . import ff8  # noqa: F401

__all__ = ["ff8"]
