"""DistillCache budgeted decode step for AMD MI355X (gfx950).

The work runs in libdistillcache.so (hand-written HIP kernels behind the C ABI
declared in include/distillcache.h); ``binding`` mirrors that ABI under the same
names and ``buffers`` allocates the device buffers with torch."""
from . import binding  # noqa: F401
