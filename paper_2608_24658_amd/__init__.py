"""Parason parallel-trajectory accounting and PA-GRPO reward on MI355X (gfx950).

The hot path is the HIP library ``libparason.so`` (C-ABI in ``include/parason.h``);
``paper_2608_24658_amd.parason`` is its Python binding.
"""
from . import parason  # noqa: F401
