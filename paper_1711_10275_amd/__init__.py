"""MI355X-native submanifold sparse convolution (SSC) and sparse convolution (SC) layers.

The hot path (coordinate dictionary, rule books, gather-MFMA-scatter forward
and backward) is hand-written HIP in ``csrc/``, built into ``libsscn.so``
and exposed through the C ABI of ``include/sscn.h``; ``sscn`` is its thin
Python binding.  ``synthetic`` draws seeded inputs.
"""
from . import sscn  # noqa: F401
