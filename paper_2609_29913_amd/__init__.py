"""MI355X-native decode attention over a block-wise low-rank KV cache.

The work runs in libmilo.so (hand-written gfx950 HIP kernels behind the C ABI
declared in include/milo.h); `milo` is a thin ctypes binding with the same
entry-point names.  Besides the decode / prefill attention it holds the
encoder's entropy rank allocation (milo_allocate_ranks).
"""
from . import milo  # noqa: F401
from .milo import (MiloError, lib, milo_allocate_ranks, milo_attend_decode, milo_attend_prefill,  # noqa: F401
                   milo_cache_create, milo_cache_device_bytes, milo_cache_free, milo_cache_read_factor,
                   milo_last_error, milo_timing_enable, milo_timing_read, milo_timing_read_alloc)
