"""CPU oracle for the ReTopK decode step -- TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The GPU library and its Python binding never do.
"""
