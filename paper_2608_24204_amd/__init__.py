"""MI355X-native dense-decoder forward (chunked prefill + batch-1 greedy decode).

The compute path is the C-ABI library ``libwici.so`` (hand-written HIP kernels for
gfx950) declared in ``include/wici.h``; :mod:`paper_2608_24204_amd.binding` is the
thin ctypes binding over it.  Importing this package loads nothing: the binding is
imported explicitly by its users, so that the configuration and input modules stay
usable on a host without a GPU.
"""

__all__ = ["configs", "inputs", "binding"]
