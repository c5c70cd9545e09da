"""DQT linear train step on MI355X (gfx950): Python side of the C-ABI library.

``dqt`` is the ctypes binding of ``libdqt.so`` (argument marshalling only);
``workloads`` holds the synthetic shapes and seeded draws.
"""
