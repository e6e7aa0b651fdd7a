"""MI355X-native decode-step state update of DAMP (arXiv 2608.27513).

The compute lives in libdamp.so (HIP kernels for gfx950 behind a C ABI, see
include/damp.h). ``paper_2608_27513_amd.damp`` is the thin ctypes binding;
``paper_2608_27513_amd.inputs`` draws seeded synthetic workloads. Importing
the package itself loads nothing native.
"""
