"""LLEP (least-loaded expert parallelism) expert-layer hot path for MI355X.

The work runs in libllep.so (HIP kernels for gfx950, C ABI in include/llep.h);
``binding`` is its ctypes binding, ``layer`` sequences the four calls,
``synth`` draws seeded synthetic inputs.
"""

from . import synth  # noqa: F401

__all__ = ["binding", "layer", "synth"]
