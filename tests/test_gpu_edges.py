"""GPU parity at the edges of the supported shapes, through the C ABI against the fp64 oracle
(bars as in tests/test_gpu_parity.py):

* the largest d_model the cache write takes (2048: 32 resident x rows fill 128 KB of LDS);
* the most outputs the packed-weight cache write takes (d_c + d_rope = 576: nine waves of 64);
* a degenerate geometry: a 1x1 latent grid, one head, 1-token chunks over a 3-token window;
* a window exactly one chunk long (every chunk replaces the whole ring and attends to itself);
* a batch of 8 small rollouts at once.
"""
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
from tests.gpu_common import (assert_attention_close, check_written_chunk,  # noqa: E402
                              host_bits, layer_for)
from tests.bf16_storage import storage_bars  # noqa: E402
from workloads import TINY, WAN, Dims, make_layer_inputs  # noqa: E402


def _write_exactness(layer, fe):
    before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
    layer.write(fe)
    stats = check_written_chunk(layer, fe, before_c, before_k)
    return sum(e for e, _ in stats) / sum(n for _, n in stats)


@pytest.mark.parametrize("mode", ["plain_weights", "packed_weights"])
def test_write_at_largest_d_model(vm, mode):
    """d_model = 2048 at Wan geometry, batch 2 (the 32-token blocks span the batch)."""
    dims = WAN.replace(d_model=2048)
    inp = make_layer_inputs(dims, seed=50, n_frames=3, batch=2)
    layer = layer_for(vm, inp, mode)
    assert _write_exactness(layer, 0) >= 0.999


def test_packed_write_at_most_outputs(vm):
    """d_c = 544, d_rope = 32: 576 outputs, nine waves of 64 outputs each (packed weights only;
    no attention kernel is built for this width, so only the write is checked)."""
    dims = WAN.replace(d_c=544)
    inp = make_layer_inputs(dims, seed=51, n_frames=3)
    layer = layer_for(vm, inp, "packed_weights")
    assert _write_exactness(layer, 0) >= 0.999


def _rollout_every_output(vm, dims, n_frames, batch, seed, modes, workgroups=(1, 0),
                          storage_bound=False):
    """Every write and every output of a rollout, each call checked on its own. storage_bound:
    each call's bars are the fixed ones or 1.5 times the error that bf16 storage alone gives on
    that call (tests/bf16_storage.py), whichever is larger, for shapes whose call yields a
    single query row (tests/test_bf16_storage.py shows that storage alone exceeds the fixed
    mean and relative-L2 bars on one call of the one-token grid)."""
    inp = make_layer_inputs(dims, seed=seed, n_frames=n_frames, batch=batch)
    for mode in modes:
        layer = layer_for(vm, inp, mode)
        exact = total = 0
        for fe in range(0, n_frames, dims.chunk_frames):
            before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
            layer.write(fe)
            for e, n in check_written_chunk(layer, fe, before_c, before_k):
                exact, total = exact + e, total + n
            for wg in workgroups:
                got = layer.attend(fe, vm.AttendOpts(n_workgroups=wg))
                for b in range(batch):
                    want = O.chunk_attention(inp, b, fe)
                    bars = storage_bars(inp, b, fe, want) if storage_bound else None
                    assert_attention_close(got[b], want, f"{mode} fe={fe} b={b} wg={wg}",
                                           bars=bars)
        assert exact / total >= 0.99, f"{exact}/{total} exactly rounded"


def test_one_token_grid(vm):
    """1x1 latent grid, one head: every chunk is a single token (one query row of a 32-row
    block) and the window holds at most 3 keys of a 32-key tile."""
    dims = Dims(d_model=64, n_heads=1, d_nope=32, d_rope=8, d_c=16, d_v=32, grid_h=1, grid_w=1,
                window_frames=3, chunk_frames=1, rope_pairs=(2, 1, 1))
    _rollout_every_output(vm, dims, n_frames=7, batch=2, seed=52,
                          modes=("plain_weights", "packed_weights"), storage_bound=True)


def test_window_of_one_chunk(vm):
    """window_frames == chunk_frames: every chunk overwrites the whole ring and attends only
    to itself."""
    dims = TINY.replace(window_frames=2, chunk_frames=2)
    _rollout_every_output(vm, dims, n_frames=6, batch=2, seed=53,
                          modes=("plain_weights", "packed_weights"))


def test_batch_of_eight(vm):
    """Eight rollouts in one call: the attention units and the write's token blocks run over
    all batch elements."""
    _rollout_every_output(vm, TINY, n_frames=4, batch=8, seed=54, modes=("packed_weights",),
                          workgroups=(3, 0))
