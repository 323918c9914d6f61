"""CPU oracle for the mixed-batch attention path and its latency model.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the benchmark's
CPU-baseline leg, never by the library or its Python binding.
"""
