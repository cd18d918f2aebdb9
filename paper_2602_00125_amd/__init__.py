"""MI355X (gfx950) hot path of the MiniTensor dense layer and broadcasting matmul.

The compute lives in the C-ABI library ``libminitensor_hip.so`` (HIP kernels in
``csrc/``, declarations in ``include/minitensor_hip.h``). ``binding`` is the thin
ctypes layer over it; ``workloads`` holds the seeded synthetic input generators.
Importing this package loads nothing; importing ``binding`` loads the library
and raises if it has not been built.
"""
__all__ = ["binding", "workloads"]
