"""GPU parity of the whole attention layer in latent form (query path absorbed into A_h, value
path into B_h, App. "Inference-Time Reparameterization") through the C ABI, against the
oracle's training-time layer (explicit per-head queries, keys and values, then W_O) in fp64.

* Tiny shape, d_q = 48 (padded to one 64-column chunk inside the packed weights), batch 2:
  every output of a 6-frame rollout, with and without a sink frame.
* Wan shape, d_q = 768 (the paper's query latent), batch 1: the chunk at frame 18 (full
  window), sampled rows.

Bars as in tests/test_gpu_parity.py, applied to y. Besides the roundings of the attention
call, this path rounds c^Q before its normalization, the packed A_h, B_h and o_lat to bf16.
"""
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
from tests.gpu_common import assert_attention_close, bf16_to_f64, dev, host_bits, sample_rows  # noqa: E402
from workloads import TINY, TINY_SINK, WAN, make_full_layer_inputs  # noqa: E402


class FullLayer:
    def __init__(self, vm, inp):
        self.vm, self.inp, d = vm, inp, inp.dims
        self.x = dev(inp.x)
        self.w_dkv, self.w_kr, self.gamma = dev(inp.w_dkv), dev(inp.w_kr), dev(inp.gamma)
        B = inp.batch
        self.c_kv = torch.zeros((B, d.window_tokens, d.d_c), dtype=torch.bfloat16, device="cuda")
        self.k_r = torch.zeros((B, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device="cuda")
        self.weights = torch.zeros(vm.layer_weights_bytes(d, inp.d_q), dtype=torch.uint8,
                                   device="cuda")
        vm.prepare_layer_weights(d, inp.d_q, dev(inp.w_dq), dev(inp.gamma_q), dev(inp.w_uq),
                                 dev(inp.w_qr), dev(inp.w_uk), dev(inp.w_uv), dev(inp.w_o),
                                 self.weights)
        self.y = torch.zeros((B, d.chunk_tokens, d.d_model), dtype=torch.bfloat16, device="cuda")

    def chunk(self, fe):
        d = self.inp.dims
        return self.x[:, fe * d.hw:(fe + d.chunk_frames) * d.hw].contiguous()

    def step(self, fe, opts=None, ws=None, write=True):
        """Cache write of the chunk (unless write=False), then videomla_attend_layer with these
        options; with a query range x and y are the range's tokens."""
        d, B = self.inp.dims, self.inp.batch
        xs = self.chunk(fe)
        if write:
            self.vm.cache_write(d, fe, B, xs, self.w_dkv, self.w_kr, self.gamma, self.c_kv,
                                self.k_r)
        if ws is None:
            ws = torch.empty(self.vm.attend_layer_workspace_bytes(d, self.inp.d_q, B, opts),
                             dtype=torch.uint8, device="cuda")
        y = self.y
        if opts is not None and (opts.query_begin or opts.query_count):
            lo, n = opts.query_begin, opts.n_queries(d)
            xs = xs[:, lo:lo + n].contiguous()
            y = torch.zeros((B, n, d.d_model), dtype=torch.bfloat16, device="cuda")
        self.vm.attend_layer(d, fe, B, self.inp.d_q, xs, self.weights, self.c_kv, self.k_r,
                             y, ws, opts=opts)
        torch.cuda.synchronize()
        return bf16_to_f64(host_bits(y))


@pytest.mark.parametrize("dims", [TINY, TINY_SINK], ids=["plain", "sink"])
def test_tiny_layer_rollout(vm, dims):
    inp = make_full_layer_inputs(dims, seed=20, n_frames=6, d_q=48, batch=2)
    layer = FullLayer(vm, inp)
    fe = 0
    while fe + dims.chunk_frames <= inp.n_frames:
        got = layer.step(fe)
        for b in range(inp.batch):
            want = O.attention_layer(inp, b, fe)
            assert_attention_close(got[b], want, f"tiny layer {dims.sink_frames} fe={fe} b={b}")
        fe = vm.window_advance(dims, fe)


def test_wan_layer_full_window(vm):
    d = WAN
    inp = make_full_layer_inputs(d, seed=21, n_frames=21, d_q=768)
    layer = FullLayer(vm, inp)
    for fe in range(0, 18, d.chunk_frames):
        xs = layer.chunk(fe)
        vm.cache_write(d, fe, 1, xs, layer.w_dkv, layer.w_kr, layer.gamma, layer.c_kv, layer.k_r)
    got = layer.step(18)
    rows = sample_rows(d.chunk_tokens, k=24, seed=18)
    want = O.attention_layer(inp, 0, 18, rows=rows)
    assert_attention_close(got[0][rows], want, "wan layer fe=18")
