"""CPU oracle for the fused attention forward path (test infrastructure only).

Nothing in the product imports this package: only the tests, the smoke check
and the benchmark's CPU-baseline leg use it.  It shares no code with the HIP
path.  Every function cites the passage of the paper it follows:

* ``attention``        -- the plain definition R = softmax(scale Q K^T) V
                          (Section 6, attention equation), float64.
* ``brute``            -- the same definition in pure-Python loops with
                          math.fsum (tiny inputs only).
* ``online``           -- the same output through per-key-tile partial
                          results (m, delta, O) folded with the associative
                          merge of Section 5.3 (the quantity a fused kernel
                          accumulates), float64; split-N folds of key ranges.
* ``tile_model``       -- the closed-formula tile derivation of Sections 4 and
                          6.2 (LDS -> KV tile, VGPR -> Q tile, CU count ->
                          grid, atom alignment).
* ``traffic``          -- closed-form HBM byte counts of Section 6.2.
"""
