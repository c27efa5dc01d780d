"""Winograd convolution with CRT-built transforms (Barabasz & Gregg, arXiv
1905.05233) for AMD MI355X (gfx950).

The computation lives in the native library ``libwinograd_crt.so`` (C ABI in
``include/winograd_crt.h``): exact-rational plan construction on the host and
hand-written HIP kernels for the kernel, input and output transforms and the
matrix-core contraction.  ``Plan`` is a thin binding over it; importing this
package does not load the library (``workloads`` is usable without it).
"""

__all__ = ["Plan", "WinogradError", "build_native"]


def __getattr__(name):
    if name == "Plan":
        from .winograd import Plan
        return Plan
    if name == "WinogradError":
        from ._native import WinogradError
        return WinogradError
    raise AttributeError(name)
