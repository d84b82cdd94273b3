"""GPU parity of the attention-sink context (one sink frame kept for good, FIFO over the other
frame slots, keys cached unrotated and rotated at window-local time) through the C ABI against
the fp64 oracle.

* Tiny sink shape (1 sink + 3 recent frames, 1-frame chunks), batch 2: every write of a
  12-frame rollout (the recent slots wrap three times) checked for slots, untouched slots and
  contents; every attention output compared, with the default and with 1, 3 and 64
  workgroups.
* Wan sink shape (1 sink + 6 recent frames = 10,920 keys, 3-frame chunks), batch 1: the chunk
  at frame 6 (the first eviction: the context is frames 0, 3..8) and the chunk at frame 237
  (context 0, 234..239: absolute temporal positions up to 239, window-local ones at most 6),
  sampled rows.

Bars as in tests/test_gpu_parity.py.
"""
import dataclasses

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
from tests.gpu_common import (Layer, assert_attention_close, check_written_chunk, dev,  # noqa: E402
                              host_bits, sample_rows)
from workloads import TINY_SINK, WAN_SINK, make_layer_inputs  # noqa: E402


def test_tiny_sink_rollout(vm):
    d = TINY_SINK
    inp = make_layer_inputs(d, seed=6, n_frames=12, batch=2)
    layer = Layer(vm, inp)
    fe = 0
    while fe + d.chunk_frames <= inp.n_frames:
        before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
        layer.write(fe)
        stats = check_written_chunk(layer, fe, before_c, before_k)
        exact = sum(e for e, _ in stats) / sum(n for _, n in stats)
        assert exact >= 0.99, exact
        for n_wg in ((0, 1, 3, 64) if fe in (4, 11) else (0,)):
            got = layer.attend(fe, vm.AttendOpts(n_workgroups=n_wg))
            for b in range(inp.batch):
                want = O.chunk_attention(inp, b, fe)
                assert_attention_close(got[b], want, f"tiny sink fe={fe} b={b} n_wg={n_wg}")
        fe = vm.window_advance(d, fe)


def test_wan_sink_first_eviction(vm):
    d = WAN_SINK
    inp = make_layer_inputs(d, seed=7, n_frames=9)
    layer = Layer(vm, inp)
    for fe in (0, 3):
        layer.write(fe)
    before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
    layer.write(6)
    stats = check_written_chunk(layer, 6, before_c, before_k)
    assert sum(e for e, _ in stats) / sum(n for _, n in stats) >= 0.999
    got = layer.attend(6)
    rows = sample_rows(d.chunk_tokens, k=24, seed=6)
    want = O.chunk_attention(inp, 0, 6, rows=rows)
    assert_attention_close(got[0][rows], want, "wan sink fe=6")


def test_wan_sink_late_in_rollout(vm):
    """Only the chunks the context needs are generated: frames 0..2 (the sink comes from the
    first chunk) and 234..239; the others stay zero in the host array and are never written."""
    d = WAN_SINK
    base = make_layer_inputs(d, seed=8, n_frames=9)          # weights, queries, 9 frames of x
    n_frames = 240
    x = np.zeros((1, n_frames * d.hw, d.d_model), np.uint16)
    x[:, 0:3 * d.hw] = base.x[:, 0:3 * d.hw]
    x[:, 234 * d.hw:240 * d.hw] = base.x[:, 3 * d.hw:9 * d.hw]
    inp = dataclasses.replace(base, x=x, n_frames=n_frames)
    layer = Layer(vm, base)                                   # ring, weights, queries on the GPU
    for fe in (0, 234, 237):
        xs = dev(x[:, fe * d.hw:(fe + d.chunk_frames) * d.hw])
        vm.cache_write(d, fe, 1, xs, layer.w_dkv, layer.w_kr, layer.gamma, layer.c_kv, layer.k_r,
                       layer.slots)
    assert O.context_frames(237, d) == [0, 234, 235, 236, 237, 238, 239]
    got = layer.attend(237)
    rows = sample_rows(d.chunk_tokens, k=24, seed=237)
    want = O.chunk_attention(inp, 0, 237, rows=rows)
    assert_attention_close(got[0][rows], want, "wan sink fe=237")
