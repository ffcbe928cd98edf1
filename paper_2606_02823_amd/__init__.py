"""MI355X-native rotated W2A4 quantized linear (Qift, arXiv 2606.02823).

* ``paper_2606_02823_amd.qift``  - ctypes binding of libqift.so (the C ABI in include/qift.h)
* ``paper_2606_02823_amd.synth`` - seeded synthetic inputs (no method arithmetic)
* ``paper_2606_02823_amd.build`` - builds libqift.so with hipcc for gfx950

Submodules are imported on demand so that importing the package pulls in
neither torch nor the HIP runtime.
"""
__version__ = "0.1"
