"""CPU oracle for PAM and PAM matrix products (test infrastructure only).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  The HIP library never does.
"""
