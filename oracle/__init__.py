"""fp64 CPU oracle of the batched multi-adapter linear layer.

Test infrastructure: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the HIP library.
"""
