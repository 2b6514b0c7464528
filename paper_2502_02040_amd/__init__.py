"""MI355X (gfx950) implementation of the M2R2 dual-stream decode path.

The compute runs in ``libm2r2.so`` (hand-written HIP kernels behind the C ABI
declared in ``include/m2r2.h``); ``binding`` marshals arguments to it.
"""
from .binding import (Model, PagedKV, M2R2Error, lib, workspace_size, EXPORTS)  # noqa: F401

__all__ = ["Model", "PagedKV", "M2R2Error", "lib", "workspace_size", "EXPORTS"]
