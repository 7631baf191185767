"""Diagonal-aware sparse decode attention for AMD Instinct MI355X (gfx950).

``libdsa.so`` (built from ``csrc/`` by ``build.py``) holds the HIP kernels and
the C ABI declared in ``include/dsa.h``; ``binding`` is its thin ctypes
binding; ``synth`` generates the seeded synthetic workloads.
"""

from . import binding  # noqa: F401
