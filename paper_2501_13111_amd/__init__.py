"""MI355X (gfx950) fingerprint forward pass: HIP kernels behind a C ABI (include/fp.h)
and a thin ctypes binding.  See ``binding.Fingerprint``."""
from .binding import Fingerprint, FpShape, FpError, fill_normal, load, lib_path  # noqa: F401
