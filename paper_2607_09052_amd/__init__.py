"""MI355X (gfx950) implementation of the COBS decode-step path.

The work happens in the HIP library libcobs.so (C ABI in include/cobs.h);
``cobs`` is its thin Python binding.
"""
from . import cobs  # noqa: F401
