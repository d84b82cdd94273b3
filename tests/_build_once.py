"""Build the HIP library once if it is not there yet (tests load what is built)."""
import importlib.util
import os

_BUILD = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "paper_2605_30351_amd", "build.py")


def _builder():
    spec = importlib.util.spec_from_file_location("videomla_build", _BUILD)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def ensure_built():
    mod = _builder()
    if not os.path.exists(mod.LIB):
        mod.build()


def ensure_stamps_built() -> str:
    """The diagnostic build (phase stamps); returns its path."""
    mod = _builder()
    if not os.path.exists(mod.STAMPS_LIB):
        mod.build(stamps=True)
    return mod.STAMPS_LIB
