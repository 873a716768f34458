"""MI355X (gfx950) expert-slot-cache MoE FFN: HIP kernels behind a C ABI.

The library is ``libmoecache.so`` (``include/moecache.h``), built in-tree by
``paper_2607_09686_amd.build``.  ``moecache`` is its ctypes binding.
"""
from .moecache import (HostBuffer, MoeCache, MoeError, SlotTable, Counters,  # noqa: F401
                       KIND_ROUTER, KIND_GATEUP, KIND_DOWN, KIND_COPY, KIND_NAMES, lib,
                       min_misses, pack_gguf, plan_bytes, plan_percent, probe_h2d,
                       probe_hbm_read)
