"""Oracle of the SoftNeuro hot path -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package; the product path (``paper_2110_06037_amd``) never imports it.

* ``numeric``: float64 layer operations and a net forward pass (C library
  ``sn_oracle.c`` plus shape bookkeeping).
* ``select``: exhaustive enumeration of routine paths (Definitions 1-2 of the
  paper) and an independent block-wise exact solver for larger nets.
"""
