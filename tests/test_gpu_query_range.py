"""GPU parity of a block of the chunk's query tokens (videomla_attend_opts query_begin /
query_count): one GPU's share of a query-sharded chunk, and the few-query regime in which the
latent cache's smaller traffic matters. The window is the whole chunk's; only the queries (and
their positions) are the block's. Each path (latent, materialized, dense comparator, whole
layer) is compared with the fp64 oracle on exactly the block's rows, at the stated tolerance
(bars as in tests/test_gpu_parity.py)."""
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
from tests.gpu_common import Layer, assert_attention_close  # noqa: E402
from workloads import SMALL, SMALL_PAPER, TINY, WAN, make_dense_inputs, make_layer_inputs  # noqa: E402

# (query_begin, query_count) over SMALL's 120-token chunk: a head block, ragged middle and tail
# blocks (none a multiple of a row block), a single token and the whole chunk (count 0)
SMALL_RANGES = ((0, 16), (37, 21), (100, 20), (119, 1), (0, 0))


def _rows(dims, lo, n):
    return np.arange(lo, lo + (n or dims.chunk_tokens - lo))


@pytest.mark.parametrize("dims,form", [(SMALL, "latent"), (SMALL_PAPER, "materialized")],
                         ids=["latent", "materialized"])
def test_small_every_output_per_range(vm, dims, form):
    """Every output row of each block, at a partial window, the exactly full window and after
    the wrap, batch 3, with 1 and the default number of workgroups."""
    inp = make_layer_inputs(dims, seed=80, n_frames=10, batch=3)
    layer = Layer(vm, inp, packed=True)
    for fe in range(0, 10, dims.chunk_frames):
        layer.write(fe)
        if fe not in (2, 4, 8):
            continue
        for lo, n in SMALL_RANGES:
            rows = _rows(dims, lo, n)
            for wg in (1, 0):
                got = layer.attend(fe, vm.AttendOpts(n_workgroups=wg, form=form, query_begin=lo,
                                                     query_count=n))
                assert got.shape[1] == len(rows)
                for b in range(inp.batch):
                    assert_attention_close(got[b], O.chunk_attention(inp, b, fe, rows=rows),
                                           f"{form} fe={fe} range=({lo},{n}) wg={wg} b={b}")


def test_tiny_sink_ranges(vm):
    """A block of queries with a sink context (window-local positions of the block's tokens)."""
    from workloads import TINY_SINK
    d = TINY_SINK
    inp = make_layer_inputs(d, seed=81, n_frames=9, batch=2)
    layer = Layer(vm, inp)
    for fe in range(9):
        layer.write(fe)
        for lo, n in ((0, 5), (7, 9), (15, 1)):
            got = layer.attend(fe, vm.AttendOpts(query_begin=lo, query_count=n))
            for b in range(2):
                assert_attention_close(got[b], O.chunk_attention(inp, b, fe, rows=_rows(d, lo, n)),
                                       f"sink fe={fe} range=({lo},{n}) b={b}")


def test_dense_comparator_ranges(vm):
    from tests.test_gpu_dense import DENSE_SMALL, DenseLayer
    d = DENSE_SMALL
    inp = make_dense_inputs(d, seed=82, n_frames=8, batch=2)
    layer = DenseLayer(vm, inp)
    for fe in range(0, 8, d.chunk_frames):
        layer.write(fe)
    for lo, n in SMALL_RANGES:
        got = layer.attend(6, vm.AttendOpts(query_begin=lo, query_count=n))
        for b in range(2):
            want = O.dense_chunk_attention(inp, b, 6, rows=_rows(d, lo, n))
            assert_attention_close(got[b], want, f"dense range=({lo},{n}) b={b}")


def test_layer_ranges(vm):
    """The whole layer with a block of the chunk's tokens as its input x and output y."""
    from tests.test_gpu_layer import FullLayer
    from workloads import make_full_layer_inputs
    d = TINY
    inp = make_full_layer_inputs(d, seed=83, n_frames=5, d_q=48, batch=2)
    layer = FullLayer(vm, inp)
    for fe in range(5):
        layer.step(fe)  # writes the chunk and attends with the whole chunk
        for lo, n in ((0, 4), (5, 7), (15, 1)):
            got = layer.step(fe, vm.AttendOpts(query_begin=lo, query_count=n), write=False)
            for b in range(2):
                want = O.attention_layer(inp, b, fe, rows=_rows(d, lo, n))
                assert_attention_close(got[b], want, f"layer fe={fe} range=({lo},{n}) b={b}")


@pytest.mark.parametrize("lo", [0, 4664], ids=["first16", "last16"])
def test_wan_sixteen_queries_batch2(vm, lo):
    """The smallest block of the few-query measurement: 16 query tokens x 12 heads per batch
    element over the wrapped 32,760-key window, batch 2; latent (even and adaptive partition,
    which splits every row block's keys over many workgroups), the automatic form choice (which
    takes the latent form here) and the dense comparator, every output row against the
    oracle."""
    d = WAN
    inp = make_layer_inputs(d, seed=84, n_frames=24, batch=2)
    layer = Layer(vm, inp, packed=True)
    for fe in range(0, 24, 3):
        layer.write(fe)
    rows = _rows(d, lo, 16)
    want = [O.chunk_attention(inp, b, 21, rows=rows) for b in range(2)]
    ws = torch.zeros(vm.attend_workspace_bytes(d, 2, vm.AttendOpts(query_count=16)),
                     dtype=torch.uint8, device="cuda")
    for part in ("even", "adaptive", "adaptive", "frozen"):
        got = layer.attend(21, vm.AttendOpts(partition=part, query_begin=lo, query_count=16),
                           ws=ws)
        for b in range(2):
            assert_attention_close(got[b], want[b], f"wan 16 queries {part} b={b}")
    auto = layer.attend(21, vm.AttendOpts(form="auto", query_begin=lo, query_count=16))
    for b in range(2):
        assert_attention_close(auto[b], want[b], f"wan 16 queries auto b={b}")
    from tests.test_gpu_dense import DenseLayer
    dinp = make_dense_inputs(d, seed=85, n_frames=24, batch=2)
    dense = DenseLayer(vm, dinp)
    for fe in range(3, 24, 3):
        dense.write(fe)
    got = dense.attend(21, vm.AttendOpts(query_begin=lo, query_count=16))
    for b in range(2):
        assert_attention_close(got[b], O.dense_chunk_attention(dinp, b, 21, rows=rows),
                               f"wan dense 16 queries b={b}")


def test_wan_auto_form_takes_the_faster_exact_form(vm):
    """form = auto on the 3-frame Wan chunk (the cost model picks the materialized form there)
    matches the oracle and the latent form; sampled rows."""
    from tests.gpu_common import sample_rows
    d = WAN
    inp = make_layer_inputs(d, seed=86, n_frames=21)
    layer = Layer(vm, inp, packed=True)
    for fe in range(0, 21, 3):
        layer.write(fe)
    assert (vm.attend_workspace_bytes(d, 1, vm.AttendOpts(form="auto"))
            == vm.attend_workspace_bytes(d, 1, vm.AttendOpts(form="materialized")))
    rows = sample_rows(d.chunk_tokens, k=16, seed=86)
    lat = layer.attend(18).copy()
    got = layer.attend(18, vm.AttendOpts(form="auto"))
    assert_attention_close(got[0][rows], O.chunk_attention(inp, 0, 18, rows=rows), "wan auto")
    assert_attention_close(got[0], lat[0], "wan auto vs latent")
