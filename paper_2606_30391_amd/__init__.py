"""MI355X-native batched energy-aware placement and migration search (Festina).

``festina`` is the ctypes binding of the C ABI in ``include/festina.h``;
``workloads`` draws seeded synthetic inputs.  Nothing is loaded at import time.
"""
__all__ = ["festina", "workloads", "build"]
