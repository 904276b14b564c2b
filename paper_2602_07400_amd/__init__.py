"""MI355X-native bit-packed LUT-network inference (BitLogic's inference path).

The compute path lives in ``libbitlogic.so`` (HIP kernels for gfx950 behind the
C ABI of ``include/bitlogic.h``); ``bitlogic`` is its Python binding and
``workloads`` draws seeded synthetic inputs.  Importing the package does not
load the shared library; the first binding call does, and raises if it is
missing.
"""
__version__ = "0.1.0"
