"""fp64 CPU oracle of the VideoMLA latent-attention path.

TEST INFRASTRUCTURE ONLY: imported by tests/, the package smoke check and the benchmark's
CPU-baseline leg, never by the product path.
"""
from .videomla_oracle import *  # noqa: F401,F403
