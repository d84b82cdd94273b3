"""GPU parity of the materialized-K/V attention (videomla_attend_ex with the materialized form:
per-head keys and values reconstructed from the latent ring, then standard attention) against the fp64
oracle, whose reference is that same training form. Bars as in tests/test_gpu_parity.py.
Both head splits it is built for: the paper's d_nope 96 + d_rope 32 (keys as wide as the
128-wide values) and d_nope 128 + d_rope 32 (160-wide keys)."""
import numpy as np
import pytest
import torch

from tests._build_once import ensure_built

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def vm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_built()
    import paper_2605_30351_amd as m
    yield m


from oracle import videomla_oracle as O  # noqa: E402
from tests.gpu_common import Layer, assert_attention_close, sample_rows  # noqa: E402
from workloads import SMALL, SMALL_PAPER, WAN, WAN_PAPER, make_layer_inputs  # noqa: E402


@pytest.mark.parametrize("dims", [SMALL_PAPER, SMALL], ids=["nope96", "nope128"])
def test_small_every_output(vm, dims):
    """Every output of a 7-chunk rollout (partial windows, ring wrap, ragged last key tile),
    batch 2, 1, 3, 7 and the default number of workgroups, against the oracle and against the
    latent path on the same ring."""
    inp = make_layer_inputs(dims, seed=60, n_frames=14, batch=2)
    layer = Layer(vm, inp, packed=True)
    for fe in range(0, 14, dims.chunk_frames):
        layer.write(fe)
        lat = layer.attend(fe)
        for wg in ((1, 3, 7, 0) if fe in (0, 6, 12) else (0,)):
            got = layer.attend(fe, vm.AttendOpts(n_workgroups=wg, form="materialized"))
            for b in range(2):
                want = O.chunk_attention(inp, b, fe)
                assert_attention_close(got[b], want, f"materialized fe={fe} b={b} wg={wg}")
                assert_attention_close(got[b], lat[b], f"materialized vs latent fe={fe} b={b}")


@pytest.mark.parametrize("dims", [WAN_PAPER, WAN], ids=["nope96", "nope128"])
def test_wan_geometry(vm, dims):
    """Wan geometry: the chunk alone (frame 0) and the wrapped 32,760-key window (frames
    3..23), sampled rows."""
    inp = make_layer_inputs(dims, seed=61, n_frames=24)
    layer = Layer(vm, inp, packed=True)
    rows = sample_rows(dims.chunk_tokens, k=24, seed=5)
    layer.write(0)
    mat = vm.AttendOpts(form="materialized")
    got = layer.attend(0, mat)
    assert_attention_close(got[0][rows], O.chunk_attention(inp, 0, 0, rows=rows), "wan fe=0")
    for fe in range(3, 22, 3):
        layer.write(fe)
    got = layer.attend(21, mat)
    assert_attention_close(got[0][rows], O.chunk_attention(inp, 0, 21, rows=rows), "wan fe=21")
