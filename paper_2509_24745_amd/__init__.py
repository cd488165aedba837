"""ProxyAttn prefill path for MI355X (gfx950).

Three HIP stages behind a C ABI (include/proxyattn.h):
proxy-head block scoring, the block-aware dynamic per-head budget with
per-head Top-K block lists, and causal block-sparse attention.

Submodules:
    proxyattn  ctypes binding of libproxyattn.so (imports torch)
    synth      seeded synthetic Q/K/V generator
    build      builds libproxyattn.so in-tree with hipcc
"""

__version__ = "0.1.0"
