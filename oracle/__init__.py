"""CPU oracle of the selective-refinement step (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path never does.
"""
from . import sphinx_oracle  # noqa: F401
from .sphinx_oracle import *  # noqa: F401,F403
