"""Pooled back-propagation for fully connected sigmoid nets on MI355X (gfx950).

The compute path is the C-ABI library ``libbp.so`` (HIP kernels, declared in
``include/bp.h``); ``paper_1801_01554_amd.bp`` is its thin ctypes binding.
Importing this package loads nothing; the binding loads the library on first
use and raises if it is missing.
"""
__all__ = ["bp", "workloads", "metrics"]
