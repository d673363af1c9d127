"""MI355X-native linear-cross-entropy (LCE): fused output projection + cross-entropy.

The compute lives in ``liblce.so`` (hand-written gfx950 HIP kernels behind a
plain C ABI, ``include/lce.h``); ``binding`` marshals arguments to it and
``autograd`` wraps the forward/backward pair as a ``torch.autograd.Function``.
Importing this package does not load the library; the first call does, and
raises if it was not built.
"""

__all__ = ["linear_cross_entropy", "LinearCrossEntropy", "AdamWState", "linear_kd_loss", "LinearKD"]


def __getattr__(name):
    if name in __all__:
        from . import autograd
        return getattr(autograd, name)
    raise AttributeError(name)
