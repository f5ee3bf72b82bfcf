"""MI355X (gfx950) W4A16 quantized linear layer: HIP kernels behind a C ABI.

``qlin`` is the Python binding of ``libqlin.so``; ``build`` compiles it.
"""
from . import qlin  # noqa: F401
from .qlin import QLinear, QlinError  # noqa: F401
