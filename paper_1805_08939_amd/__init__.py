"""Approximate Random Dropout (arXiv 1805.08939) hot path for MI355X (gfx950).

The computation lives in libard.so (C ABI, include/ard.h): pattern search and
sampling on the host, compaction and the fwd / bwd_data / bwd_weight GEMMs of
FC, tile-pattern and LSTM layers on the GPU. ``api`` is the same-name Python
binding; ``synth`` builds seeded synthetic workloads.
"""

from . import api  # noqa: F401
from ._ffi import LIB_PATH  # noqa: F401
