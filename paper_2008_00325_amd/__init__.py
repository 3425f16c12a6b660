"""MI355X-native layout SGD of GPU UMAP (Nolet et al., AAAI 2021).

The compute path is the C-ABI library ``libumap_layout.so`` built from
``csrc/`` (hand-written HIP for gfx950); ``umap_layout`` is its ctypes
binding and ``synth`` the seeded workload generators.
"""
