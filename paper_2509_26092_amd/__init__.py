"""MI355X (gfx950) ResNet-18 training step and dual-batch parameter-server
merge, as hand-written HIP kernels behind a C ABI (include/rn18.h).

``binding`` holds the ctypes binding (same names as the C ABI); ``inputs``
the seeded synthetic input generators; ``build`` compiles the library.
"""
from . import binding  # noqa: F401
