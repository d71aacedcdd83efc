"""OrderMoE layer path for AMD Instinct MI355X (gfx950).

The compute lives in libordermoe.so (HIP kernels + host C++, C ABI in
include/ordermoe.h); `ordermoe` is its ctypes binding.
"""
from . import ordermoe  # noqa: F401
