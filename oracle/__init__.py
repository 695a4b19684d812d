"""Float64 CPU oracle for the spectral spin-weighted spherical convolution.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link anything in this package; only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` use it.  It shares no code with the GPU path: the two meet only
at the seeded input generators, which hold none of the method's arithmetic.
"""

from .swsft_oracle import *  # noqa: F401,F403
