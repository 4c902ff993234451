"""Float64 CPU oracle of the KronQ per-layer path.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may import this package. The product path (the HIP library and its Python
binding) never imports, calls or falls back to it, and shares no code with it.
"""
from .kronq_oracle import *  # noqa: F401,F403
from .kronq_oracle import __all__  # noqa: F401
