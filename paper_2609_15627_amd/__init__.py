"""MI355X (gfx950) routed mixture-of-experts layer: HIP kernels behind a C ABI.

The kernels live in csrc/*.hip and are built into libmoe.so by ``_build``;
``moe`` is the thin ctypes binding (importing it requires the built library).
"""
import os

PACKAGE_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PACKAGE_DIR, "libmoe.so")
