"""Oracle: plain, slow, obviously correct CPU restatements of what the GPU
path computes. TEST INFRASTRUCTURE ONLY: imported by tests, by the smoke
check and by the benchmark's CPU-baseline leg, never by the product.

  gemm_ref.c / gemm_ref.py  C = A * B in fp64 from bf16/fp16 inputs
  grouped_ref.py            the grouped product (one plain product per
                            group of consecutive rows, per-group B)
  taxonomy.py               the tiling taxonomy and the latency model's
                            closed forms, in exact rational arithmetic

Parity status: every function here is pinned by tests against values the
paper prints, closed forms, invariants or brute force (see the tests named
test_oracle_*). One quantity is not pinned: the absolute accuracy of the
calibrated cost constants (the paper does not print them) -- parity unpinned;
the tests check the model's formulas, not its constants.
"""
