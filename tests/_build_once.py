"""Build the HIP library once if it is not there yet (tests load what is built)."""
import importlib.util
import os

_BUILD = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "paper_2605_30351_amd", "build.py")


def ensure_built():
    spec = importlib.util.spec_from_file_location("videomla_build", _BUILD)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    if not os.path.exists(mod.LIB):
        mod.build()
