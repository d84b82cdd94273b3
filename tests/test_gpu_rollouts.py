"""GPU parity over longer schedules of the calls, through the C ABI against the fp64 oracle.

* Denoising steps and layers: several cache_write + attend pairs at one window position
  overwrite the same slots (each step's chunk activations differ); each layer has its own
  weights and ring; after the window advance the next chunk evicts the oldest frames.
  Wan geometry, two layers, four steps at frame 18, then frame 21.
* Rollout: batch 4, 80 consecutive 3-frame chunks (frames 0..239): the ring wraps eleven times
  and temporal positions reach 239. Spot checks at chunk 0 (the window is the chunk alone),
  chunk 6 (the first full window) and chunk 79, for batch elements 0 and 3, plus the slots of
  every chunk. The chunk activations are drawn on the GPU from a seeded torch generator (one
  per chunk) and copied to the host for the oracle.

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
from workloads import WAN, f32_to_bf16_bits, make_layer_inputs  # noqa: E402


def test_denoising_steps_overwrite_then_advance(vm):
    d = WAN
    hw = d.hw
    for layer_seed in (3, 33):  # two layers: own weights, own ring
        inp = make_layer_inputs(d, seed=layer_seed, n_frames=24)  # final activations per frame
        layer = Layer(vm, inp)
        for fe in range(0, 18, 3):
            layer.write(fe)
        rows = sample_rows(d.chunk_tokens, k=8, seed=layer_seed)
        rng = np.random.default_rng(1000 + layer_seed)
        n_steps = 4
        for step in range(n_steps):
            x_step = inp.x.copy()
            if step < n_steps - 1:  # earlier denoising steps see other chunk activations
                draw = rng.standard_normal((1, d.chunk_frames * hw, d.d_model), dtype=np.float32)
                x_step[:, 18 * hw:21 * hw] = f32_to_bf16_bits(draw)
            layer.inp = dataclasses.replace(inp, x=x_step)
            layer.x = dev(x_step)
            before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
            layer.write(18)
            stats = check_written_chunk(layer, 18, before_c, before_k)
            exact = sum(e for e, _ in stats) / sum(n for _, n in stats)
            assert exact >= 0.999, exact
            got = layer.attend(18)
            if step in (0, n_steps - 1):
                want = O.chunk_attention(layer.inp, 0, 18, rows=rows)
                assert_attention_close(got[0][rows], want,
                                       f"layer seed {layer_seed} step {step} at frame 18")
        fe = vm.window_advance(d, 18)
        assert fe == 21
        layer.inp, layer.x = inp, dev(inp.x)
        layer.write(fe)
        got = layer.attend(fe)
        want = O.chunk_attention(inp, 0, fe, rows=rows)  # frames 3..23; 0..2 evicted
        assert_attention_close(got[0][rows], want, f"layer seed {layer_seed} after advance")


def test_rollout_batch4_eighty_chunks(vm):
    d = WAN
    hw, B, n_chunks = d.hw, 4, 80
    inp = make_layer_inputs(d, seed=4, n_frames=d.chunk_frames, batch=B)  # weights, queries
    layer = Layer(vm, inp)

    def chunk_x(c):
        g = torch.Generator(device="cuda")
        g.manual_seed(40_000 + c)
        return torch.randn((B, d.chunk_tokens, d.d_model), generator=g, device="cuda",
                           dtype=torch.float32).to(torch.bfloat16)

    checked = (0, 6, n_chunks - 1)
    check_b = (0, 3)
    rows = sample_rows(d.chunk_tokens, k=6, seed=4)
    fe = 0
    for c in range(n_chunks):
        assert fe == d.chunk_frames * c
        vm.cache_write(d, fe, B, chunk_x(c), layer.w_dkv, layer.w_kr, layer.gamma, layer.c_kv,
                       layer.k_r, layer.slots)
        n = np.arange(d.chunk_tokens)
        f, y, x = O.token_position(n, fe, d)
        assert np.array_equal(layer.slots.cpu().numpy(), O.ring_slot(f, y, x, d).astype(np.int32))
        if c in checked:
            got = layer.attend(fe)
            lo, hi = O.window_frame_range(fe, d)
            # frames 0 .. hi-1 in the oracle's layout; only the window's frames are filled (the
            # zeros of np.zeros are not touched, so the untouched part costs no memory)
            x_host = np.zeros((B, hi * hw, d.d_model), np.uint16)
            for cc in range(lo // d.chunk_frames, hi // d.chunk_frames):
                bits = host_bits(chunk_x(cc))
                for b in check_b:
                    x_host[b, cc * d.chunk_frames * hw:(cc + 1) * d.chunk_frames * hw] = bits[b]
            ref_inp = dataclasses.replace(inp, x=x_host, n_frames=hi)
            for b in check_b:
                want = O.chunk_attention(ref_inp, b, fe, rows=rows)
                assert_attention_close(got[b][rows], want, f"rollout chunk {c} (frame {fe}) b={b}")
        fe = vm.window_advance(d, fe)
