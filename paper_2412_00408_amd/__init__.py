"""libquake: QuAKE (arXiv:2412.00408) exp approximation fused into Softmax,
GELU and Logistic, as hand-written HIP kernels for MI355X (gfx950).

The C ABI is declared in include/quake.h and implemented in csrc/; the
ctypes binding with the same names lives in `paper_2412_00408_amd.quake`
(imported lazily so that the seeded input generators in `synth` can be used
without the built library).
"""

__all__ = ["quake", "synth"]


def __getattr__(name):
    if name == "quake":
        from . import quake as _q
        return _q
    if name == "synth":
        from . import synth as _s
        return _s
    raise AttributeError(name)
