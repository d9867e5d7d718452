"""MI355X-native fused WTConv (wavelet convolution) forward and backward.

The compute path is the C-ABI library ``libwtconv.so`` (hand-written gfx950
HIP kernels, declared in ``include/wtconv.h``). This package holds its thin
Python binding (:mod:`.binding`), an autograd wrapper (:mod:`.autograd`), the
seeded synthetic input generator (:mod:`.inputs`) and the I/O accounting
(:mod:`.iomodel`). Submodules are imported lazily so that host-only users
(tests of the input generator, the accounting) need neither torch nor a GPU.
"""
__all__ = ["binding", "autograd", "inputs", "iomodel"]
