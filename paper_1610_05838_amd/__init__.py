"""MI355X-native SGD matrix factorisation (the hot path of arXiv 1610.05838).

The GPU work lives in ``libmfsgd.so`` (HIP, gfx950) behind a C ABI declared in
``include/mfsgd.h``; ``paper_1610_05838_amd.mfsgd`` is the thin ctypes binding.
Importing this package loads nothing: the binding loads the library on first
use and raises if it has not been built.
"""
