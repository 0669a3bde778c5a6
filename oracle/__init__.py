"""fp64 CPU oracle for segment-local non-causal softmax attention.

Test infrastructure only: the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package; the product path (the HIP library and its binding) never imports it.
"""
