"""CPU oracle of the GDP policy forward pass and sampling (float64 numpy).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg; never by the product path.
"""
