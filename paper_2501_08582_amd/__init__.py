"""Sparsity-preserved LoRA linear (LoRS, arXiv 2501.08582) for AMD MI355X.

The compute lives in ``liblors.so`` (hand-written HIP kernels for gfx950 behind
the C ABI in ``include/lors.h``).  Python modules:

``ops``    PyTorch-facing calls and the autograd op (imports torch)
``_lib``   ctypes binding of the C ABI
``synth``  seeded synthetic inputs shaped like the paper's Llama projections
``costs``  flop / byte accounting
``build``  hipcc build of ``liblors.so``
"""

__all__ = ["ops", "synth", "costs", "build"]
__version__ = "1.0.0"
