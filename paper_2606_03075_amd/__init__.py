"""TGV-KV eviction pass and pruned-cache decode for MI355X (gfx950).

The computation lives in libtgvkv.so (hand-written HIP kernels behind the C ABI
of include/tgvkv.h); ``binding`` marshals torch device tensors to it.
"""

__all__ = ["binding", "build"]
