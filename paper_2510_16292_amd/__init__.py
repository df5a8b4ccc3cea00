"""QSVD latent-QKV hot path for AMD Instinct MI355X (gfx950).

* :mod:`.binding` -- ctypes binding of the C ABI in ``include/qsvd.h``
  (``libqsvd.so``, built by :mod:`.build`).
* :mod:`.prep` -- the offline stage: joint SVD, beta split and weight
  quantization into the layout the library consumes.
"""
from . import prep  # noqa: F401
