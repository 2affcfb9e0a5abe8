"""libquake: QuAKE (arXiv:2412.00408) exp approximation fused into Softmax,
GELU and Logistic, as hand-written HIP kernels for MI355X (gfx950).

The C ABI is declared in include/quake.h and implemented in csrc/; the ctypes
binding with the same names is the submodule `paper_2412_00408_amd.quake`
(import it explicitly; it raises if libquake.so is not built). The seeded
synthetic workloads are in `paper_2412_00408_amd.synth`.
"""
