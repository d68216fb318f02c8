"""MI355X-native fused routed-MoE decode operator (MonoMoE, arXiv 2609.04244).

The operator is one persistent HIP kernel for gfx950 behind the C ABI in
include/monomoe.h; ``monomoe`` is its ctypes binding, ``workloads`` the seeded
synthetic input generator.
"""
