"""MI355X-native DeRF renderer (Voronoi-decomposed radiance fields).

The compute path lives in the HIP library ``libderf.so`` (C ABI declared in
``include/derf.h``); ``paper_2011_12490_amd.derf`` is its thin ctypes
binding.  Importing the package loads nothing native.
"""
