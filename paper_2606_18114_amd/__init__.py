"""Grouped-absmean ternary (W1.58A16) linear layer for AMD MI355X (gfx950).

The compute path is ``libtmamba.so`` (hand-written HIP kernels behind the C
ABI declared in ``include/tmamba.h``); ``ops`` is a thin ctypes binding that
marshals torch tensors into those calls; ``qat`` wires them into autograd
as the TernaryLinear layer.  ``synth`` draws the seeded synthetic inputs.  Importing the package does not load the library; the
first call into ``ops`` does, and raises if it has not been built.
"""

__all__ = ["ops", "qat", "synth"]
