"""fp64 CPU oracle for the block-quantized linear layer (test infrastructure).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never does.
"""
