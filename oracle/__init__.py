"""CPU oracle for BSR pruning and BSR x dense products.

TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the CPU-baseline timing leg of
the benchmark.  It never imports the library package and shares no code with it.
"""
