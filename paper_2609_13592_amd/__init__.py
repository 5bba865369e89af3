"""MI355X-native tiered-memory (HBM + pinned host) decode path.

The compute path is the HIP library ``_lib/libboostcap.so`` (built by
``paper_2609_13592_amd.build``); ``binding`` marshals arguments to its C-ABI.
There is no CPU fallback: loading fails loudly when the library is missing.
"""
from .binding import (  # noqa: F401
    BoostError, lib_path, load,
)
