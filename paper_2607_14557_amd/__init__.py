"""Seer hot path on MI355X (gfx950): C-ABI library libseer.so + thin binding.

The library (include/seer.h) holds the HIP kernels: the bidirectional layer
over packed variable-length sequences with the fused near-zero activation
count, the SNR boundary scan, and routing + compaction.  ``seer`` is the
ctypes binding (same names as the C ABI); ``runner`` sequences the calls.
"""
from . import seer
from .seer import load_library, SeerError
