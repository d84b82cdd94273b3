"""GPU parity of the paper's d_c sweep (Table 5: latent widths 64, 128, 192, 256 and 512 with
the 32-wide RoPE key) and of the few-query regime (1-frame chunks), through the C ABI against
the fp64 oracle. Bars as in tests/test_gpu_parity.py. At d_c = 512 the attention splits the
value columns over wave pairs and only the packed-weight cache write applies (544 outputs)."""
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
from tests.gpu_common import (Layer, assert_attention_close, check_written_chunk,  # noqa: E402
                              host_bits, sample_rows)
from workloads import SMALL, WAN_1F, WAN_DC, make_layer_inputs  # noqa: E402

SWEEP = (64, 128, 256, 512)  # 192 is the default shape, covered by the other parity tests


@pytest.mark.parametrize("d_c", SWEEP)
def test_small_every_output(vm, d_c):
    """Every write and every output of a 7-chunk rollout (ring wraps; last key tile ragged),
    batch 2, packed and plain weights, 1, 3 and the default number of workgroups."""
    dims = SMALL.replace(d_c=d_c)
    inp = make_layer_inputs(dims, seed=20 + d_c, n_frames=14, batch=2)
    for packed in ((True,) if d_c + dims.d_rope > 288 else (False, True)):
        layer = Layer(vm, inp, packed=packed)
        exact = total = 0
        for fe in range(0, 14, dims.chunk_frames):
            before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
            layer.write(fe)
            for e, n in check_written_chunk(layer, fe, before_c, before_k):
                exact, total = exact + e, total + n
            for wg in ((1, 3, 0) if fe in (0, 6, 12) else (0,)):
                got = layer.attend(fe, vm.AttendOpts(n_workgroups=wg))
                for b in range(2):
                    assert_attention_close(got[b], O.chunk_attention(inp, b, fe),
                                           f"d_c={d_c} packed={packed} fe={fe} b={b} wg={wg}")
        assert exact / total >= 0.999, f"{exact}/{total} exactly rounded"


@pytest.mark.parametrize("d_c", SWEEP)
def test_wan_geometry_full_window(vm, d_c):
    """Wan geometry at this latent width: the write that evicts frames 0..2 and the attention
    of the chunk of frames 21..23 over the wrapped 32,760-key window (sampled rows)."""
    dims = WAN_DC[d_c]
    inp = make_layer_inputs(dims, seed=30 + d_c, n_frames=24)
    layer = Layer(vm, inp, packed=True)
    for fe in range(0, 19, 3):
        layer.write(fe)
    before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
    layer.write(21)
    stats = check_written_chunk(layer, 21, before_c, before_k)
    assert sum(e for e, _ in stats) / sum(n for _, n in stats) >= 0.999
    got = layer.attend(21)
    rows = sample_rows(dims.chunk_tokens, k=24, seed=d_c)
    assert_attention_close(got[0][rows], O.chunk_attention(inp, 0, 21, rows=rows),
                           f"wan d_c={d_c}")


def test_wan_one_frame_chunks(vm):
    """Few-query regime: 1-frame chunks (1,560 queries x 12 heads per call), batch 2, at the
    rollout start (the chunk alone), with an exactly full window (frames 0..20) and after
    the ring has wrapped (frames 2..22)."""
    dims = WAN_1F
    inp = make_layer_inputs(dims, seed=40, n_frames=23, batch=2)
    layer = Layer(vm, inp, packed=True)
    rows = sample_rows(dims.chunk_tokens, k=24, seed=3)
    rows = rows[rows < dims.chunk_tokens]
    for fe in range(23):
        layer.write(fe)
        if fe in (0, 20, 22):
            got = layer.attend(fe)
            for b in ((0, 1) if fe == 22 else (0,)):
                assert_attention_close(got[b][rows], O.chunk_attention(inp, b, fe, rows=rows),
                                       f"1-frame chunks fe={fe} b={b}")
