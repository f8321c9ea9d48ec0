"""Oracle of the two-phase VLA forward (fp64 NumPy).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; never by the product path.
It shares no code with the HIP library (only the seeded input generator
``synth`` serves both sides).
"""
from .vla_oracle import *  # noqa: F401,F403
from .vla_oracle import forward, vlm_prefill, action_denoise  # noqa: F401
