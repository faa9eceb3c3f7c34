"""ELIS hot path on MI355X: iterative remaining-length prediction + ISRTF selection.

The compute lives in libelis.so (HIP, gfx950), declared in include/elis.h.
``_elis`` is the ctypes binding (same names as the C entry points);
``device`` keeps weights and workspaces in HBM through PyTorch allocations;
``driver`` packs scheduling rounds and calls the two entry points.
"""
from . import _elis  # noqa: F401
