"""MI355X-native KV-offload data path (EfficientAgent, arXiv 2609.33762).

The library (libea.so, C ABI in include/ea.h) moves paged KV cache state
between HBM and a pinned host tier with hand-written HIP kernels for gfx950,
computes chained SHA-256 prefix-block keys on the GPU, and keeps the LRU host
tier with its working-set-aware write admission on the CPU.

`api` holds the Python binding; `workloads` the seeded synthetic inputs.
The shared library is loaded on first use, not at import.
"""
__all__ = ["api", "workloads"]
