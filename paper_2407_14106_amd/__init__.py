"""Graph-topology sparse attention (TorchGT, arXiv 2407.14106) for AMD MI355X.

The compute lives in ``libgt.so`` (HIP kernels for gfx950 behind the C ABI of
``include/gt.h``); ``gt`` is its ctypes binding.  Import is cheap: the library
is loaded on first use (``load()``), and loading fails loudly when it is not
built.
"""

from __future__ import annotations


def load():
    """Load libgt.so and return the binding module."""
    from . import gt

    gt.load_library()
    return gt
