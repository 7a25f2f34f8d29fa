"""fp64 CPU oracle for the verification and distillation path (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never does.
"""
