"""CPU oracle for the NITRO-D integer training step.

Test infrastructure only: imported by the tests, the smoke check and the CPU-baseline leg of the
benchmark, never by the product path.
"""
