"""Shared-prefix continuous-sampling decode attention for MI355X (gfx950).

The compute path is the C-ABI library ``libinfs.so`` (HIP kernels + host
runtime + refill scheduler, see ``include/infs.h``); ``infs`` is its ctypes
binding and ``group`` drives one group decode through it.
"""

__all__ = ["infs", "group"]
