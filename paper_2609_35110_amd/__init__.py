"""MI355X-native fused 3D-RoPE + softmax attention (video DiT self-attention).

The compute lives in ``libsol.so`` (HIP kernels for gfx950 behind a C ABI,
declared in ``include/sol.h``); this package is the thin Python binding over
it plus the seeded workload generator.
"""
