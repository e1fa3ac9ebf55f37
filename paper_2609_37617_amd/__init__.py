"""MI355X (gfx950) target verification step of AS2D (arXiv 2609.37617).

The compute path is the HIP library libas2d.so (csrc/), declared in
include/as2d.h; `as2d` is its thin ctypes binding.
"""
