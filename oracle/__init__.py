"""CPU oracle for the SubZero+ hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, float64 NumPy written from the paper (SubZero+, arXiv 2608.15665):
Eq. 4 (per-query subspace perturbation), Eqs. 5-6 and Alg. 3 (query losses and
the estimate), Eqs. 7-10 (subspace Adam), Eq. 11 and Alg. 1 (Haar QR with sign
correction), Alg. 2 (perturbation of the weights).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path:
the only module both sides use is ``zo_draws`` (seeded inputs, no method
arithmetic).  Nothing here is ever a fallback for the GPU path.
"""
from .subzero import *  # noqa: F401,F403
