"""MI355X (gfx950) batched kernel-latency evaluator of KernelSight-LM.

The product is libks.so (HIP kernels + C ABI, include/ks.h); ``abi`` is its
thin ctypes binding."""

__all__ = ["abi", "build"]
