"""Locks per-step sparse decode attention for AMD MI355X (gfx950).

The compute path lives in the HIP library liblocks.so (C ABI: include/locks.h);
`paper_2607_24555_amd.locks` is its ctypes binding.
"""
from . import locks  # noqa: F401
from .locks import (Config, LocksError, build_factors, build_summaries,  # noqa: F401
                    decode_step, dense_attend, select, sparse_attend, workspace_bytes)
