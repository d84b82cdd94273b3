"""GPU parity of the weighted (per-XCD) work partition of the attention kernels.

In adaptive mode every call re-splits the units from the previous adaptive call's per-XCD
times, kept in a state area at the end of the attention workspace (bal_prep_kernel sets the
weights, the attention kernel records each workgroup's duration), so consecutive calls on one
workspace use different split points. Frozen mode reuses the weights the state holds and
records nothing. Each call is checked against the fp64 oracle on sampled rows and, on every row,
against the even split of the same inputs (bars as in tests/test_gpu_parity.py: the two differ
only in rounding). Every path (latent, whole layer, dense comparator, materialized form) must
leave a valid state record after adaptive calls, so that a silent fallback to the even split
fails here.
"""
import numpy as np
import pytest
import torch

from tests._build_once import ensure_built

pytestmark = pytest.mark.gpu

BAL_HEAD, BAL_MAX_WG = 16, 4096
BAL_WORDS = BAL_HEAD + BAL_MAX_WG                   # one state area
BAL_BYTES = (BAL_WORDS * 4 + 255) // 256 * 256      # its place in the workspace
BAL_MIN, BAL_MAX, BAL_MARK = 820, 1280, 0x564D4C42


@pytest.fixture(scope="module")
def vm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_built()
    import paper_2605_30351_amd as m
    yield m


from oracle import videomla_oracle as O  # noqa: E402
from tests.gpu_common import Layer, assert_attention_close, sample_rows  # noqa: E402
from workloads import TINY, WAN, make_layer_inputs  # noqa: E402


def _state(ws, end=None):
    """The partition state area that ends at byte `end` of the workspace (default: its end)."""
    torch.cuda.synchronize()
    end = ws.numel() if end is None else end
    return ws[end - BAL_BYTES:end - BAL_BYTES + BAL_WORDS * 4].cpu().numpy().view(np.uint32)


def _assert_recorded(st, label):
    """A state written by an adaptive call: marker, G, weights in range, every duration set."""
    assert st[9] == BAL_MARK, f"{label}: no partition record (the call did not run adaptive)"
    G = int(st[8])
    assert 1 <= G <= BAL_MAX_WG, (label, G)
    assert np.all((st[:8] >= BAL_MIN) & (st[:8] <= BAL_MAX)), (label, st[:8])
    assert np.all(st[BAL_HEAD:BAL_HEAD + G] > 0), f"{label}: a workgroup recorded no duration"
    return G


def test_wan_adaptive_then_frozen(vm):
    inp = make_layer_inputs(WAN, seed=31, n_frames=24)
    layer = Layer(vm, inp)
    for fe in range(0, 24, 3):
        layer.write(fe)
    ws = torch.zeros(vm.attend_workspace_bytes(WAN, 1), dtype=torch.uint8, device="cuda")
    even = layer.attend(21, ws=ws)
    rows = sample_rows(WAN.chunk_tokens, k=16, seed=31)
    want = O.chunk_attention(inp, 0, 21, rows=rows)
    assert_attention_close(even[0][rows], want, "even split")
    assert _state(ws)[9] != BAL_MARK, "the even split leaves no record"
    # frozen before any adaptive call: equal weights, i.e. the even split, bit for bit
    got = layer.attend(21, vm.AttendOpts(partition="frozen"), ws=ws)
    assert np.array_equal(got, even)
    adaptive = vm.AttendOpts(partition="adaptive")
    for call in range(4):
        got = layer.attend(21, adaptive, ws=ws)
        assert_attention_close(got[0][rows], want, f"adaptive call {call} vs oracle")
        assert_attention_close(got[0], even[0], f"adaptive call {call} vs even split")
        G = _assert_recorded(_state(ws), f"adaptive call {call}")
        assert G == 256 or G == torch.cuda.get_device_properties(0).multi_processor_count
    st = _state(ws).copy()
    frozen = vm.AttendOpts(partition="frozen")
    fa = layer.attend(21, frozen, ws=ws).copy()
    fb = layer.attend(21, frozen, ws=ws)
    assert np.array_equal(fa, fb), "frozen calls are bitwise reproducible"
    assert np.array_equal(_state(ws), st), "frozen calls leave the state as it was"
    assert_attention_close(fa[0][rows], want, "frozen vs oracle")


def test_two_workspaces_keep_their_own_record(vm):
    """Two workspaces used alternately (A, B, A, B): each call reads and writes only its own
    workspace's state, so both hold a complete record."""
    inp = make_layer_inputs(WAN, seed=36, n_frames=21)
    layer = Layer(vm, inp, packed=True)
    for fe in range(0, 21, 3):
        layer.write(fe)
    size = vm.attend_workspace_bytes(WAN, 1)
    wa = torch.zeros(size, dtype=torch.uint8, device="cuda")
    wb = torch.zeros(size, dtype=torch.uint8, device="cuda")
    adaptive = vm.AttendOpts(partition="adaptive")
    rows = sample_rows(WAN.chunk_tokens, k=8, seed=36)
    want = O.chunk_attention(inp, 0, 18, rows=rows)
    for call in range(2):
        for name, ws in (("A", wa), ("B", wb)):
            got = layer.attend(18, adaptive, ws=ws)
            assert_attention_close(got[0][rows], want, f"workspace {name} call {call}")
            _assert_recorded(_state(ws), f"workspace {name} call {call}")


def test_adaptive_mode_on_small_shapes_and_partitions(vm):
    """Tiny rollout (every output) in adaptive and frozen mode with several workgroup counts:
    shapes whose ranges would get too short keep the even split, larger counts of units take
    the weighted one; every output matches the oracle either way."""
    inp = make_layer_inputs(TINY, seed=32, n_frames=6, batch=2)
    layer = Layer(vm, inp)
    for fe in range(6):
        layer.write(fe)
        for wg in (1, 3, 0):
            ws = torch.zeros(vm.attend_workspace_bytes(TINY, 2, vm.AttendOpts(n_workgroups=wg)),
                             dtype=torch.uint8, device="cuda")
            for part in ("adaptive", "adaptive", "frozen"):
                got = layer.attend(fe, vm.AttendOpts(n_workgroups=wg, partition=part), ws=ws)
                for b in range(inp.batch):
                    assert_attention_close(got[b], O.chunk_attention(inp, b, fe),
                                           f"tiny fe={fe} b={b} wg={wg} {part}")


def test_wan_layer_adaptive_calls(vm):
    """The whole layer (its latent merge reads the weighted split points) on two consecutive
    adaptive calls, sampled rows against the oracle; the record sits at the end of the layer
    workspace's attention part."""
    from tests.test_gpu_layer import FullLayer
    from workloads import make_full_layer_inputs
    d = WAN
    inp = make_full_layer_inputs(d, seed=33, n_frames=21, d_q=768)
    layer = FullLayer(vm, inp)
    for fe in range(0, 18, d.chunk_frames):
        xs = layer.chunk(fe)
        vm.cache_write(d, fe, 1, xs, layer.w_dkv, layer.w_kr, layer.gamma, layer.c_kv, layer.k_r)
    rows = sample_rows(d.chunk_tokens, k=12, seed=33)
    want = O.attention_layer(inp, 0, 18, rows=rows)
    adaptive = vm.AttendOpts(partition="adaptive")
    ws = torch.zeros(vm.attend_layer_workspace_bytes(d, 768, 1, adaptive), dtype=torch.uint8,
                     device="cuda")
    att_end = vm.attend_workspace_bytes(d, 1, adaptive)
    for call in range(2):
        got = layer.step(18, adaptive, ws=ws)
        assert_attention_close(got[0][rows], want, f"adaptive layer call {call}")
        _assert_recorded(_state(ws, att_end), f"adaptive layer call {call}")


def test_dense_and_materialized_adaptive_calls(vm):
    """The dense comparator and the materialized form in adaptive mode (their merges read the
    weighted split points): two consecutive calls each at Wan geometry, sampled rows, and the
    record each leaves in its own workspace."""
    from tests.test_gpu_dense import DenseLayer
    from workloads import make_dense_inputs
    d = WAN
    rows = sample_rows(d.chunk_tokens, k=16, seed=34)
    dinp = make_dense_inputs(d, seed=34, n_frames=21)
    dense = DenseLayer(vm, dinp)
    for f in range(0, 21, d.chunk_frames):
        dense.write(f)
    want_d = O.dense_chunk_attention(dinp, 0, 18, rows=rows)
    inp = make_layer_inputs(d, seed=35, n_frames=21)
    layer = Layer(vm, inp, packed=True)
    for f in range(0, 21, d.chunk_frames):
        layer.write(f)
    want_m = O.chunk_attention(inp, 0, 18, rows=rows)
    d_opts = vm.AttendOpts(partition="adaptive")
    m_opts = vm.AttendOpts(partition="adaptive", form="materialized")
    ws_d = torch.zeros(vm.dense_attend_workspace_bytes(d, 1, d_opts), dtype=torch.uint8,
                       device="cuda")
    ws_m = torch.zeros(vm.attend_workspace_bytes(d, 1, m_opts), dtype=torch.uint8, device="cuda")
    for call in range(2):
        got = dense.attend(18, d_opts, ws=ws_d)
        assert_attention_close(got[0][rows], want_d, f"adaptive dense call {call}")
        _assert_recorded(_state(ws_d), f"adaptive dense call {call}")
        got = layer.attend(18, m_opts, ws=ws_m)
        assert_attention_close(got[0][rows], want_m, f"adaptive materialized call {call}")
        _assert_recorded(_state(ws_m), f"adaptive materialized call {call}")
