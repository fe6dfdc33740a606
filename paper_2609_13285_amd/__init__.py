"""MI355X-native decode-step attention of Grouped Value Attention (GVA).

The compute path lives in ``libgva.so`` (hand-written HIP for gfx950 behind a
C ABI, declared in ``include/gva.h``).  ``paper_2609_13285_amd.gva`` is the
thin ctypes binding with the same entry-point names; importing this package
loads nothing, and the first call into the binding raises if the library is
missing.
"""

__all__ = ["gva", "traffic"]
