"""KVBoost's stitched-prefill path on one AMD Instinct MI355X (gfx950).

* ``kvb``       -- ctypes binding of ``lib/libkvb.so`` (the C ABI of ``include/kvb.h``)
* ``pipeline``  -- builds the path's inputs in HBM and runs the path through the ABI
* ``trace``     -- a synthetic request trace shaped like the paper's workload, run
  request by request (``python -m paper_2608_21362_amd.trace``)
* ``build``     -- compiles ``csrc/`` with hipcc for gfx950 (and ``ceiling/``, the
  practical-ceiling kernels the benchmark measures)

``kvb`` is imported on first use so that ``build`` runs before the library exists.
"""
__all__ = ["kvb", "pipeline", "trace", "build"]
