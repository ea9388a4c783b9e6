"""CPU oracle for the LayerCheck decision step (test infrastructure only).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
use it; the HIP library never imports or links anything from here.
"""
