"""fp64 CPU oracle — TEST INFRASTRUCTURE ONLY.

This package is the reference the tests check against, never part of the product path. Only the tests,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it. It shares no code with the HIP library or its Python binding; the
only thing both sides consume is the seeded input generator in ``synth``.

Modules:
  layer       plain numpy float64 definition of the dense GQA decoder layer,
              its stages, the 80-layer model head and greedy argmax.
  bruteforce  an independent scalar-loop version of the same layer for tiny
              shapes (pure Python floats, no numpy arithmetic).
"""
from . import layer, bruteforce  # noqa: F401
