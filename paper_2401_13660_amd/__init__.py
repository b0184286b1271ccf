"""MI355X-native selective scan (the S6 scan at the heart of every MambaByte layer).

The compute path is the HIP library ``libmbscan.so`` (hand-written gfx950
kernels behind a C ABI declared in ``include/mbscan.h``); this package is a thin
binding over it.  ``scan_fwd`` (and ``scan_fwd_noalloc``, the same scan with nothing allocated),
``scan_step``, the backward ``scan_bwd``, the causal
convolution upstream
of the scan, ``conv1d`` and ``conv1d_step``, and the top-beta check that ends a
speculative verification, ``verify_rank``, are loaded on first use.
``selective_scan`` is the scan as a differentiable torch operation (forward with
checkpoints, backward from them).
"""
__all__ = ["scan_fwd", "scan_fwd_noalloc", "scan_step", "scan_bwd", "conv1d", "conv1d_step", "verify_rank", "load_library",
           "MBScanError", "selective_scan"]


def __getattr__(name):
    if name == "selective_scan":
        from .autograd import selective_scan
        return selective_scan
    if name in __all__:
        from . import _binding
        return getattr(_binding, name)
    raise AttributeError(name)
