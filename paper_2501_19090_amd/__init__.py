"""MI355X-native PIFA (Pivoting Factorization) layer forward.

The compute path is ``libpifa.so`` (hand-written HIP for gfx950 behind a C
ABI, declared in ``include/pifa.h``); :mod:`paper_2501_19090_amd.pifa` is the
thin ctypes binding.  Importing the package loads nothing: the library is
opened on first use, and every entry point raises if it is missing.
"""
