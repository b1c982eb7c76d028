"""Plain CPU oracle of the SFS TTFT estimator and the latency-aware router.

TEST INFRASTRUCTURE ONLY.  Imported by the tests, the smoke check and the CPU
baseline leg of the benchmark; never by the product path.
"""
