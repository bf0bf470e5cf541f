"""MI355X-native training hot path of parareal neural networks (Lee, Lee & Park).

``binding`` is the thin ctypes layer over ``libpnn.so`` (C ABI in ``include/pnn.h``);
``step`` strings the entry points together into one training step (Alg. para2 then Alg. para3)
on device buffers allocated through PyTorch.
"""
from . import binding  # noqa: F401
