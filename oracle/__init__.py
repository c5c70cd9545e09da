"""CPU oracle for the DQT linear train step.

TEST INFRASTRUCTURE, NOT PRODUCT CODE: only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with the HIP library.
"""
from .dqt_oracle import *  # noqa: F401,F403
