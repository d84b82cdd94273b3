"""GPU parity of the cache write's less common branches, against the fp64 oracle (Eq. 1 with
the RMSNorm of the latent, Eq. 5, and the ring placement of App. "Chunk-Causal Sliding-Window
Attention"): a gain that is not all ones, no gain at all, and a cache with an attention sink
(keys kept unrotated, Sec. "Decoupled 3D-RoPE"), each through the packed kernel (up to 32 tokens
per compute unit), the wide kernel (batched calls, one workgroup per compute unit) and the
plain-weight kernel. Slots are compared bit-exact, untouched ring rows must keep their bits,
and the written rows must be within one bf16 step of the oracle (check_written_chunk)."""
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


from tests.gpu_common import Layer, check_written_chunk, host_bits  # noqa: E402
from workloads import WAN, WAN_SINK, make_layer_inputs  # noqa: E402


def _check_chunk(layer, fe, min_exact=0.999):
    before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
    layer.write(fe)
    stats = check_written_chunk(layer, fe, before_c, before_k)
    exact = sum(e for e, _ in stats) / sum(n for _, n in stats)
    print(f"fe={fe}: {exact:.5f} of the written values exact", flush=True)
    assert exact >= min_exact


# batch 1: the packed kernel (19 tokens per compute unit); batch 2: the wide kernel (37)
@pytest.mark.parametrize("batch,packed", [(1, True), (2, True), (2, False)])
def test_wan_write_with_random_gain(vm, batch, packed):
    """A gain drawn uniform in [0.5, 1.5): each latent output must take its own entry."""
    inp = make_layer_inputs(WAN, seed=41, n_frames=6, batch=batch, random_gain=True)
    assert len(np.unique(inp.gamma)) > 100
    layer = Layer(vm, inp, packed=packed)
    _check_chunk(layer, 0)
    _check_chunk(layer, 3)


@pytest.mark.parametrize("batch", [1, 2])
def test_wan_write_without_gain(vm, batch):
    """No RMSNorm: the latents are stored as projected."""
    inp = make_layer_inputs(WAN, seed=42, n_frames=3, batch=batch, norm=False)
    assert inp.gamma is None
    layer = Layer(vm, inp, packed=True)
    _check_chunk(layer, 0)


@pytest.mark.parametrize("batch", [1, 2])
def test_wan_sink_write_keeps_keys_unrotated(vm, batch):
    """With a sink frame the keys are cached unrotated, in the sink-aware slots: the write of
    frames 6..8 into a 7-frame window (1 sink + 6 cycling slots) fills the last free slot and
    evicts frames 1 and 2, keeping frame 0."""
    inp = make_layer_inputs(WAN_SINK, seed=43, n_frames=9, batch=batch, random_gain=True)
    layer = Layer(vm, inp, packed=True)
    for fe in (0, 3):
        _check_chunk(layer, fe)
    _check_chunk(layer, 6)
