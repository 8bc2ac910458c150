"""Paged decode attention for AMD MI355X (gfx950).

The compute path is the HIP library ``_lib/libpda.so`` (sources in ``csrc/``,
C ABI in ``include/pda.h``); ``binding`` marshals torch tensors into it.
"""
from . import binding  # noqa: F401
from .binding import paged_decode_attention, plan, workspace_reserve  # noqa: F401
