"""MI355X (gfx950) prover for the Range-Arithmetic protocol: sum-check over
multilinear extensions for fixed-point matrix products, plus concatenated
range-proof sum-checks for rounding and ReLU.

Import ``paper_2505_17623_amd.ra`` for the C-ABI binding (loads the HIP
library) and ``paper_2505_17623_amd.inputs`` for seeded synthetic workloads.
"""
__all__ = ["ra", "inputs"]
