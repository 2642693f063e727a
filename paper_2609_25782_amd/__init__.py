"""Hot-cold KV-cache hot path for AMD Instinct MI355X (gfx950).

``hotcold_kv`` is the ctypes binding of the C ABI (``include/hotcold_kv.h``);
``pool.HotColdPool`` wraps a pool whose buffers are torch tensors.  Importing
``hotcold_kv`` fails if the HIP library has not been built
(``python -m paper_2609_25782_amd.build``).
"""

__all__ = ["hotcold_kv", "pool", "build"]
