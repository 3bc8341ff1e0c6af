"""CPU oracle of the stitched-prefill path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, readable restatement of what KVBoost's stitched-prefill step
computes, in float64 numpy, written from the paper (KVBoost, arXiv 2608.21362):

* ``rope``       -- rotary position embedding and its position correction
                    (Sec. 3.2, Eq. 3)
* ``kivi``       -- KIVI asymmetric quantisation, keys per channel, values per
                    token (Sec. 4.5, Eq. 7 and the sentence after it)
* ``stitch``     -- dequantise cached chunks and re-rotate keys to their new
                    position (Sec. 4.3 prompt assembly, Sec. 3.2)
* ``deviation``  -- CacheBlendRecompute step 2 (Alg. 2)
* ``selection``  -- CacheBlendRecompute step 3 (Alg. 2) united with the
                    SelectiveRecompute seam windows (Alg. 1) and live rows
                    (Sec. 4.1 attention sinks, Sec. 4.7 live tokens)
* ``attention``  -- CacheBlendRecompute step 4 patch (Alg. 2) and causal
                    attention of the selected query rows (Sec. 3.1, Eq. 2)
* ``populate``   -- turns the seeded raw draws of ``kvb_workload`` into the
                    rotated / quantised inputs the path consumes

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The HIP library and its Python binding
never import, call or link anything here, and nothing here imports them.
"""
