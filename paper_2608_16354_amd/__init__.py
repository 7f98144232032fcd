"""DriveCache cache-aware denoising step on MI355X (gfx950).

The compute lives in libdrivecache.so (hand-written HIP kernels + the host
schedule behind a C ABI, include/dc.h); `api` is its Python binding and
`inputs` generates seeded synthetic workloads.
"""
from . import inputs  # noqa: F401

__all__ = ["inputs", "api"]
