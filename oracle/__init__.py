"""fp64 CPU oracle of the ST-Lite compression pass (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  It shares no code with the HIP library.
"""
