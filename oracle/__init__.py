"""CPU oracle for Eq. (1) of the HPTT paper.

TEST INFRASTRUCTURE, NOT PRODUCT CODE: only the test-suite, the smoke check of
the entry module and the CPU-baseline leg of the benchmark may import it.
"""
