"""MI355X-native streaming equivariant tensor-product convolution (arXiv 2607.18074).

The operator runs in libsobek_hip.so (C ABI, generated HIP kernels for gfx950);
this package holds the thin Python binding (``_lib``, ``api``), the build
script and the seeded workload generators.
"""
