"""CPU oracle for the attention path (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg
may import this package.  The HIP library never does.
"""
