"""liblpv: the block-sparse linear layer Y = g(X W~^T + b) of LPViT
(arXiv 2407.02068) for AMD MI355X.

The compute path is the HIP library ``liblpv.so`` (C ABI in include/lpv.h);
:mod:`paper_2407_02068_amd.lpv` is its thin ctypes binding.
"""
from .lpv import (BsrWeight, LpvError, bsr_export, bsr_info, bsr_linear, bsr_pack,  # noqa: F401
                  bsr_schedule_export, bsr_unpack, dense_linear, last_error, lib, status_str)
