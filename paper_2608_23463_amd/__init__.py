"""MI355X-native ProxyFormer hot path: the HIP library and its Python binding.

Submodules (imported on demand so that importing the package needs no GPU):
  binding - ctypes binding of libproxyformer.so (the C ABI)
  synth   - seeded synthetic inputs shaped like the paper's workloads
  build   - builds libproxyformer.so for gfx950
"""
