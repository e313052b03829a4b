"""CPU oracle for the LookME hot path.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package; the library and its binding never do.

  lookme_oracle  plain float64 implementation of the paper's definitions
  brute          pure-Python loops with exact rational arithmetic (tiny inputs)
  check          tie- and rounding-aware comparison of library outputs
"""
