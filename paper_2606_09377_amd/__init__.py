"""vcrown: batched CROWN bound propagation for ReLU networks on AMD MI355X (gfx950).

The bounds are computed by the HIP kernels of lib/libvcrown.so (C ABI in
include/vcrown.h); `vcrown.Ctx` is a thin ctypes binding over it.
"""
from .vcrown import Ctx, VcrError, load_library, header_symbols  # noqa: F401
