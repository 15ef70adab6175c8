"""CHAOS oracle: a plain CPU implementation used only as test infrastructure.

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
it.  It shares no code with the HIP library (paper_1506_09067_amd).
"""
