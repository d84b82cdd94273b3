"""The diagnostic build (libvideomla_stamps.so, include/videomla_stamps.h) computes the same
outputs as the product library, bit for bit, and records every named point of every
workgroup in order.

The binding picks its library at import, so the diagnostic build runs in a child process
(tests/stamps_child.py) on the same seeded inputs as this process's product run
(tests/stamps_run.py): one Wan2.1-1.3B chunk-step (packed cache write, attend on the even
split) and one batch-4 cache write (the wide kernel)."""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

from tests._build_once import ensure_built, ensure_stamps_built

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def vm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_built()
    ensure_stamps_built()
    import paper_2605_30351_amd as m
    if m.STAMPS:
        pytest.skip("this process loaded the diagnostic build")
    yield m


def test_stamps_build_matches_product_and_records_in_order(vm, tmp_path):
    from tests.stamps_run import run
    want = run(vm)
    env = dict(os.environ, VIDEOMLA_LIBRARY="stamps")
    print("child: tests/stamps_child.py (diagnostic build)", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "stamps_child.py"),
                        str(tmp_path)], env=env, cwd=ROOT, capture_output=True, text=True,
                       timeout=240)
    print(r.stdout)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    for name, t in want.items():
        got = np.load(tmp_path / (name + ".npy"))
        assert np.array_equal(got, t.numpy()), f"{name} differs between the two builds"
