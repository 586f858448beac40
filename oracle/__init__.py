"""CPU oracle for exact top-k context-sparse decode attention.

Test infrastructure only: the tests, the package smoke check and the
benchmark's CPU-baseline leg may use it; the product path never does.
"""
