"""Oracle: plain CPU reference implementations used to check the HIP engine.

TEST INFRASTRUCTURE ONLY. The product path (paper_2606_03014_amd) never
imports this package; only tests/, the package smoke check and the benchmark's
CPU-baseline leg do.
"""
