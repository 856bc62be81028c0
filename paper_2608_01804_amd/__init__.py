"""MI355X (gfx950) hot path of LEAP's GRPO training step (arXiv 2608.01804).

``paper_2608_01804_amd.leap`` is the ctypes binding of ``libleap.so`` (HIP
kernels + C ABI declared in ``include/leap.h``); build it with
``paper_2608_01804_amd._build.build()``.  Importing this package loads
nothing; the library is opened on first use and its absence raises.
"""
from . import leap  # noqa: F401

__all__ = ["leap"]
