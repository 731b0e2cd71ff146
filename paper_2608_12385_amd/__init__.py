"""Decode-Branch Transformer grouped decode on MI355X (gfx950).

The compute path is libdbt.so (HIP kernels behind the C ABI in
include/dbt.h); ``binding`` marshals arguments to it through ctypes.
"""
from . import binding  # noqa: F401
from .binding import DbtError, Session  # noqa: F401
