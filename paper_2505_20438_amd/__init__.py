"""HAMburger macro-step decode loop on AMD MI355X (gfx950).

The compute lives in ``libham.so`` (HIP kernels behind the C ABI declared in
``include/ham.h``); :mod:`paper_2505_20438_amd.ham` is its ctypes binding.
Importing this package has no side effects.
"""
