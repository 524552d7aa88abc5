"""fp64 CPU oracle for the DTST spectral-layer path.

Test infrastructure only: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``, never by the library.
"""
from .dtst_oracle import *  # noqa: F401,F403
from .dtst_oracle import __all__  # noqa: F401
