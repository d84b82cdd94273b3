"""Build the HIP library once if it is not there yet (tests load what is built)."""
import os

from paper_2605_30351_amd import build as _build


def ensure_built():
    if not os.path.exists(_build.LIB):
        _build.build()
