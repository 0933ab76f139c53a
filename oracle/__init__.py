"""CPU oracle of the Federation-of-Experts per-cluster MoE block.

Test infrastructure only: imported by the tests, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py``, never by the product path.
"""
from .foe_oracle import *  # noqa: F401,F403
from .foe_oracle import __all__  # noqa: F401
