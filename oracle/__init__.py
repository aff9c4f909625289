"""CPU oracle of the routing simulation: test infrastructure only.

Used by the test suite, the smoke check and the CPU-baseline leg of the
benchmark.  The product path never imports this package.
"""
