"""CPU oracle for the Flash-BoN batched draft step (fp64, numpy).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py``; never by the library or its binding.  See ``oracle/dit.py`` for what it follows.
"""
from . import dispatch, dit, phi, sde  # noqa: F401
