"""fp64 CPU oracle for the hybrid causal-attention layer (test infrastructure
only: the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may use it; the GPU product path never does)."""

from .saf_oracle import *  # noqa: F401,F403
from .saf_oracle import __all__  # noqa: F401
