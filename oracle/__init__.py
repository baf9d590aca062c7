"""Plain CPU fp64 reference for SPHQuant's decode path.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import it. The library and its HIP kernels never call it, and it
imports nothing from the library.
"""
from . import sph  # noqa: F401
