"""rat3d: MI355X-native training step of a 3D residual attention network.

The compute lives in ``librat3d.so`` (hand-written HIP for gfx950 behind a C
ABI declared in ``include/rat3d.h``).  ``paper_2104_05035_amd.rat3d`` is the
thin ctypes binding; ``paper_2104_05035_amd.synth`` makes seeded synthetic
inputs.  Importing the package loads nothing.
"""
