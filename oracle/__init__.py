"""CPU oracle for the PEFT-BD speculative step -- TEST INFRASTRUCTURE ONLY.

Plain, slow, float64 NumPy code that states what the hot path computes, for
the tests, the package smoke check and the benchmark's CPU baseline.  The
product path (the HIP library and its Python binding) never imports, links or
executes anything under ``oracle/``, and nothing here imports the product.

Modules:
  model  -- cached forward, prefill, draft, verify, accept, commit, generate
  brute  -- no-cache brute-force decoder with explicit masks (pins ``model``)

Every function is pinned by a CPU test (tests/test_oracle_*.py); none is
"parity unpinned".
"""
from . import model, brute  # noqa: F401
