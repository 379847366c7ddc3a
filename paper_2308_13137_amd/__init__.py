"""MI355X-native OmniQuant block-wise calibration step.

The compute path lives in ``liboq.so`` (HIP kernels for gfx950 behind a C
ABI, declared in ``include/oq.h``); :mod:`paper_2308_13137_amd.oq` is the thin
ctypes binding.  Importing this package loads nothing: the binding loads the
library on first use and raises if it is missing.
"""
