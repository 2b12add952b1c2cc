"""CPU oracle for the exact Euclidean distance transform, the brute-force
transform under three metrics and the chamfer transform.

Test infrastructure only: the tests, the smoke check and the benchmark's
CPU-baseline leg use it to check and time the GPU library.  The GPU library
never imports it, and it imports nothing from the GPU library.
"""
