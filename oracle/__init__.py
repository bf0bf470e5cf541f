"""Test infrastructure: the fp64 CPU oracle of the parareal neural network.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may import,
call or build anything under ``oracle/``.  The product path never does; it shares no code with
this package.
"""
