"""MI355X (gfx950) implementation of DuoGPT's layer-wise calibration solver.

The compute lives in libduo.so (hand-written HIP, C ABI in include/duo.h);
`duo` is its thin Python binding.
"""

from . import duo  # noqa: F401
from .duo import prune_linear  # noqa: F401
