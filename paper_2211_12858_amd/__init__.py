"""MI355X-native sketched multioutput split search (SketchBoost hot path).

The compute path is libsketchboost.so (hand-written HIP for gfx950) behind
the C ABI in include/sb.h.  ``_lib`` is the thin ctypes binding with the same
names as the C calls; ``driver`` allocates device buffers with torch and
strings the calls together.  There is no CPU fallback: importing ``_lib``
without the built library raises.
"""
