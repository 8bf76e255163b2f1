"""MI355X-native single-launch transformer decode step (arXiv 2609.12379's hot path).

The compute path is the HIP library ``libfm.so`` behind the C ABI in ``include/fm.h``;
``fm.py`` is its ctypes binding, ``metrics.py`` the Eq. 2 / Eq. 3 byte accounting.
"""
