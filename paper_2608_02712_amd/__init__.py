"""MI355X (gfx950) validation and failure-forensics library.

The engine-owned validator of the paper's debug loop: candidate operator
outputs are compared with reference outputs over every test case (tolerance
gate, NaN/Inf counts, exact max abs/rel error, error sums, per-tile mismatch
map, ordered first-k mismatch indices, degenerate-output detectors, suite
match rates), in hand-written HIP kernels behind the C ABI of
include/vcheck.h. This package is the thin Python binding; see vcheck.py.
"""
from .vcheck import (  # noqa: F401
    FLAG_ALL_ZERO, FLAG_CONSTANT, FLAG_INPUT_COPY, FLAG_LOWPREC_BF16, FLAG_LOWPREC_FP16,
    Sweep, VcheckError, compare, integrity, lib, localize, sweep, vcheck_compare,
    vcheck_integrity, vcheck_localize, vcheck_sweep, vcheck_tile_count, vcheck_workspace_bytes)
