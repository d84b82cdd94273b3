"""GPU parity of the dense per-head comparator (full-head 3D RoPE keys and values, standard
softmax attention over the same window) through the C ABI against the fp64 oracle.

* Small shape, batch 2: 2 heads of 128, a 6x10 grid, a 5-frame window (300 keys: nine whole
  32-key tiles and a ragged one) and 2-frame chunks (120 query rows per head, padded to one
  256-row block). Every output is compared; the ring contents and slots after each write too.
* Wan shape, batch 1: 12 heads of 128 at the 30x52 grid, 21-frame window. The chunk at frame 0
  (the window is the chunk alone: 4,680 keys, a ragged last tile) and at frame 18 (the first
  full window, 32,760 keys), on sampled rows that include frame and row borders.

Bars as for the latent path: bf16 outputs within max-abs 2e-2 and mean-abs 2e-3 of the fp64
result (or 8 and 4 bf16 units of the output's scale when that is larger), relative L2 1e-2;
ring values within one bf16 step of the exactly rounded result; slots bit-exact.
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
from tests.gpu_common import (SENTINEL, assert_attention_close, bf16_to_f64, dev,  # noqa: E402
                              host_bits, sample_rows, ulp_distance)
from workloads import WAN, make_dense_inputs  # noqa: E402

DENSE_SMALL = WAN.replace(d_model=128, n_heads=2, grid_h=6, grid_w=10, window_frames=5,
                          chunk_frames=2)


class DenseLayer:
    """Device copies of the comparator's inputs plus its ring [B][ring][H][2 d_v]."""

    def __init__(self, vm, inp):
        self.vm, self.inp, d = vm, inp, inp.dims
        self.x = dev(inp.x)
        self.w_k, self.w_v, self.q = dev(inp.w_k), dev(inp.w_v), dev(inp.q)
        B = inp.batch
        self.kv = torch.full((B, d.window_tokens, d.n_heads, 2 * d.d_v), SENTINEL,
                             dtype=torch.int16, device="cuda").view(torch.bfloat16)
        self.slots = torch.full((d.chunk_tokens,), -1, dtype=torch.int32, device="cuda")
        self.out = torch.zeros((B, d.chunk_tokens, d.n_heads, d.d_v), dtype=torch.bfloat16,
                               device="cuda")

    def write(self, fe):
        d = self.inp.dims
        xs = self.x[:, fe * d.hw:(fe + d.chunk_frames) * d.hw].contiguous()
        self.vm.dense_cache_write(d, fe, self.inp.batch, xs, self.w_k, self.w_v, self.kv,
                                  self.slots)

    def attend(self, fe, opts=None, ws=None):
        """videomla_dense_attend with these options (None: the defaults), into a fresh workspace
        unless `ws` is given; with a query range the queries and outputs are the range's."""
        d = self.inp.dims
        B = self.inp.batch
        if ws is None:
            ws = torch.empty(self.vm.dense_attend_workspace_bytes(d, B, opts), dtype=torch.uint8,
                             device="cuda")
        q, out = self.q, self.out
        if opts is not None and (opts.query_begin or opts.query_count):
            lo, n = opts.query_begin, opts.n_queries(d)
            q = q[:, lo:lo + n].contiguous()
            out = torch.zeros((B, n, d.n_heads, d.d_v), dtype=torch.bfloat16, device="cuda")
        self.vm.dense_attend(d, fe, B, q, self.kv, out, ws, opts=opts)
        torch.cuda.synchronize()
        return bf16_to_f64(host_bits(out))


def check_dense_chunk(layer, fe, before):
    """Slots bit-exact, other slots untouched, K and V within one bf16 step."""
    inp, d = layer.inp, layer.inp.dims
    torch.cuda.synchronize()
    kv = host_bits(layer.kv)
    slots = layer.slots.cpu().numpy()
    exact_frac = []
    for b in range(inp.batch):
        ref = O.dense_cache_write(inp.x[b, fe * d.hw:(fe + d.chunk_frames) * d.hw], inp.w_k,
                                  inp.w_v, fe, d)
        assert np.array_equal(slots, ref["slots"].astype(np.int32))
        written = np.zeros(d.window_tokens, bool)
        written[ref["slots"]] = True
        assert np.array_equal(kv[b][~written], before[b][~written])
        rows = kv[b][ref["slots"]]                       # [T, H, 2 d_v]
        for got, exact in ((rows[..., :d.d_v], ref["k"]), (rows[..., d.d_v:], ref["v"])):
            dist = ulp_distance(got, O.round_to_bf16_bits(exact))
            floor = 2.0 ** -16 * np.sqrt(np.mean(exact * exact, axis=-1, keepdims=True))
            near = np.abs(bf16_to_f64(got) - exact) <= floor
            bad = (dist > 1) & ~near
            assert not bad.any(), f"{bad.sum()} elements beyond 1 ulp; max distance {dist.max()}"
            exact_frac.append(np.count_nonzero(dist == 0) / dist.size)
    assert min(exact_frac) >= 0.99, exact_frac


def test_dense_small_every_output(vm):
    d = DENSE_SMALL
    inp = make_dense_inputs(d, seed=11, n_frames=8, batch=2)
    layer = DenseLayer(vm, inp)
    checked = 0
    for fe in range(0, 8, d.chunk_frames):
        if fe + d.chunk_frames > inp.n_frames:
            break
        before = host_bits(layer.kv)
        layer.write(fe)
        check_dense_chunk(layer, fe, before)
        got = layer.attend(fe)
        for b in range(inp.batch):
            want = O.dense_chunk_attention(inp, b, fe)
            assert_attention_close(got[b], want, f"dense small fe={fe} b={b}")
            checked += 1
    assert checked == 8


@pytest.mark.parametrize("fe", [0, 18])
def test_dense_wan_sampled_rows(vm, fe):
    d = WAN
    inp = make_dense_inputs(d, seed=5, n_frames=fe + d.chunk_frames)
    layer = DenseLayer(vm, inp)
    lo, _ = O.window_frame_range(fe, d)
    for f in range(lo, fe, d.chunk_frames):
        layer.write(f)
    before = host_bits(layer.kv)
    layer.write(fe)
    check_dense_chunk(layer, fe, before)
    got = layer.attend(fe)
    rows = sample_rows(d.chunk_tokens, k=24, seed=fe)
    want = O.dense_chunk_attention(inp, 0, fe, rows=rows)
    assert_attention_close(got[0][rows], want, f"dense wan fe={fe}")


def test_dense_split_keys_match_single_pass(vm):
    """The stream-K partial results merge exactly: many workgroups (every row block's keys
    split over several of them) against one workgroup per row block, on the same ring."""
    d = DENSE_SMALL
    inp = make_dense_inputs(d, seed=12, n_frames=6, batch=2)
    layer = DenseLayer(vm, inp)
    for fe in (0, 2, 4):
        layer.write(fe)
    outs = [layer.attend(4, vm.AttendOpts(n_workgroups=n_wg)) for n_wg in (1, 2, 7, 64)]
    want = O.dense_chunk_attention(inp, 1, 4)
    for o in outs:
        assert_attention_close(o[1], want, "dense split")
        assert np.abs(o - outs[0]).max() <= 2 * 2.0 ** -8 * np.abs(outs[0]).max()
