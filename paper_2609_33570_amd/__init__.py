"""HiLoRe hot path on AMD Instinct MI355X (gfx950).

The compute lives in libhilore.so (hand-written HIP kernels behind the C-ABI
of include/hilore.h); ``hilore`` is its thin ctypes binding and ``workloads``
draws the seeded synthetic inputs.
"""
from . import workloads  # noqa: F401

__all__ = ["defaults", "hilore", "workloads"]
