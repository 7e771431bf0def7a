"""CPU oracle for the STaR-Quant W4A4 hot path.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
anything from this package.  It shares no code with the HIP library.
"""
