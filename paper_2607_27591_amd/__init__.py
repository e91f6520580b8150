"""MI355X-native Prox sparse SwiGLU FFN decode step (HIP for gfx950).

The compute path lives in ``csrc/`` and is exported by ``libprox.so`` through
the C-ABI declared in ``include/prox.h``; ``prox`` is the thin ctypes binding.
"""
