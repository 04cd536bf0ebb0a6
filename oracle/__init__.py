"""CPU oracle for the bf16x3 compensated GEMM (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its binding) never
does, and the two share no code.
"""
