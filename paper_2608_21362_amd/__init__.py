"""KVBoost's stitched-prefill path on one AMD Instinct MI355X (gfx950).

* ``kvb``       -- ctypes binding of ``lib/libkvb.so`` (the C ABI of ``include/kvb.h``)
* ``pipeline``  -- builds the path's inputs in HBM and runs the path through the ABI
* ``build``     -- compiles ``csrc/`` with hipcc for gfx950

``kvb`` is imported on first use so that ``build`` runs before the library exists.
"""
__all__ = ["kvb", "pipeline", "build"]
