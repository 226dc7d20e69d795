"""Oracle for the BD-LoRA shard forward -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct CPU implementation (numpy, float64) of what
one tensor-parallel shard computes in block-diagonal LoRA serving.  Only the
test-suite, the smoke check and the benchmark's CPU-baseline leg may import
it; the product path (the HIP library and its Python binding) never does, and
this package imports nothing from the product path.

Modules:

* :mod:`oracle.bdlora`  -- the shard forward (Alg. 1 and Alg. 2 of the paper),
  full-matrix BD-LoRA with explicit block-diagonal factors (Sec. 3), the
  compact storage and slicing of block-diagonal factors (App. C.2), the merged
  single-adapter form (Sec. 1 reparametrisation), and a pure-Python brute
  force for tiny inputs.
* :mod:`oracle.plan`    -- id validation and grouping of tokens by adapter.
* :mod:`oracle.costs`   -- the parameter, operation and byte counts of the
  paper's cost table (App. A).
* :mod:`oracle.mlp`     -- the MLP shard of Alg. 1 (two projections with the
  activation between them).
* :mod:`oracle.quant`   -- the INT4 base weight (weight-only quantized base of
  Sec. 5.2): decoding of the stored nibbles and scales.

Every function is pinned by tests under ``tests/`` against facts the paper or
plain mathematics fixes; see each module's header for its pins.
"""
from . import bdlora, plan, costs, mlp, quant  # noqa: F401
