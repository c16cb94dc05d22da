"""MI355X-native FP8 linear-layer hot path: amax, FP8 quantisation and scaled
FP8 GEMMs (Fprop, Dgrad, Wgrad) as hand-written HIP for gfx950 behind a C ABI
(``include/puro.h``), with a thin ctypes binding in ``paper_2608_27370_amd.puro``.
"""
