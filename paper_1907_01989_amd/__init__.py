"""mgi: MobileNet-class convolutional network inference on MI355X (gfx950).

The engine is the C-ABI library libmgi.so (include/mgi.h); this package holds
its sources (csrc/), the build step (build_lib) and a ctypes binding with the
same entry-point names (_binding) plus a small torch front end (engine).
"""
from . import _binding
from ._binding import MgiError

__all__ = ["_binding", "MgiError"]
