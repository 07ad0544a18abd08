"""CPU oracle of the WISE hot path — test infrastructure only.

Imported only by the tests, the smoke check and the benchmark's CPU-baseline
leg.  Never imported by the library or its binding.
"""
