"""GPU parity of the adaptive (per-XCD) work partition of the latent attention.

In adaptive mode every call re-splits the units from the previous call's per-XCD times, so
consecutive calls on one workspace use different split points. Each call is checked against
the fp64 oracle on sampled rows and, on every row, against the even split of the same inputs
(bars as in tests/test_gpu_parity.py: the two differ only in rounding). The state record the
calls leave in the workspace must hold weights within the documented range.
"""
import numpy as np
import pytest
import torch

from tests._build_once import ensure_built

pytestmark = pytest.mark.gpu

BAL_SLOT_WORDS = 16 + 4096  # header words + per-workgroup durations, per state slot
BAL_MIN, BAL_MAX, BAL_MARK = 820, 1280, 0x564D4C42


@pytest.fixture(scope="module")
def vm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ensure_built()
    import paper_2605_30351_amd as m
    yield m
    m.set_attend_balance(False)
    m.set_attend_workgroups(0)


from oracle import videomla_oracle as O  # noqa: E402
from tests.gpu_common import (Layer, assert_attention_close, bf16_to_f64,  # noqa: E402
                              host_bits, sample_rows)
from workloads import TINY, WAN, make_layer_inputs  # noqa: E402


def _state_slots(ws):
    """The two state slots at the end of an attention workspace, as uint32 words."""
    size = (2 * BAL_SLOT_WORDS * 4 + 255) // 256 * 256
    words = ws[-size:].cpu().numpy().view(np.uint32)
    return words[:BAL_SLOT_WORDS], words[BAL_SLOT_WORDS:2 * BAL_SLOT_WORDS]


def _attend(vm, layer, fe, ws):
    d = layer.inp.dims
    vm.attend(d, fe, layer.inp.batch, layer.q_nope, layer.q_r, layer.w_uk, layer.w_uv,
              layer.c_kv, layer.k_r, layer.out, ws)
    torch.cuda.synchronize()
    return bf16_to_f64(host_bits(layer.out))


def test_wan_adaptive_calls_match_oracle_and_even_split(vm):
    inp = make_layer_inputs(WAN, seed=31, n_frames=24)
    layer = Layer(vm, inp)
    for fe in range(0, 24, 3):
        layer.write(fe)
    ws = torch.empty(vm.attend_workspace_bytes(WAN, 1), dtype=torch.uint8, device="cuda")
    even = _attend(vm, layer, 21, ws)
    rows = sample_rows(WAN.chunk_tokens, k=16, seed=31)
    want = O.chunk_attention(inp, 0, 21, rows=rows)
    assert_attention_close(even[0][rows], want, "even split")
    vm.set_attend_balance(True)
    try:
        for call in range(4):
            got = _attend(vm, layer, 21, ws)
            assert_attention_close(got[0][rows], want, f"adaptive call {call} vs oracle")
            assert_attention_close(got[0], even[0], f"adaptive call {call} vs even split")
        marked = [s for s in _state_slots(ws) if s[9] == BAL_MARK]
        assert len(marked) == 2, "both state slots written"
        for s in marked:
            assert np.all((s[:8] >= BAL_MIN) & (s[:8] <= BAL_MAX)), s[:8]
            G = int(s[8])
            assert 1 <= G <= 4096
            assert np.all(s[16:16 + G] > 0), "every workgroup recorded its duration"
    finally:
        vm.set_attend_balance(False)


def test_adaptive_mode_on_small_shapes_and_partitions(vm):
    """Tiny rollout (every output) in adaptive mode with several workgroup counts: shapes whose
    ranges would get too short keep the even split, larger counts of units take the adaptive
    one; every output matches the oracle either way."""
    inp = make_layer_inputs(TINY, seed=32, n_frames=6, batch=2)
    layer = Layer(vm, inp)
    vm.set_attend_balance(True)
    try:
        for fe in range(6):
            layer.write(fe)
            for wg in (1, 3, 0):
                vm.set_attend_workgroups(wg)
                for _ in range(2):
                    got = layer.attend(fe)
                    for b in range(inp.batch):
                        assert_attention_close(got[b], O.chunk_attention(inp, b, fe),
                                               f"tiny fe={fe} b={b} wg={wg}")
    finally:
        vm.set_attend_workgroups(0)
        vm.set_attend_balance(False)


def test_wan_layer_adaptive_calls(vm):
    """The whole layer (its latent merge reads the adaptive split points) on two consecutive
    adaptive calls, sampled rows against the oracle."""
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
    vm.set_attend_balance(True)
    try:
        for call in range(2):
            got = layer.step(18)
            assert_attention_close(got[0][rows], want, f"adaptive layer call {call}")
    finally:
        vm.set_attend_balance(False)


def test_dense_and_materialized_adaptive_calls(vm):
    """The dense comparator and the materialized form in adaptive mode (their merge reads the
    adaptive split points): two consecutive calls each at Wan geometry, sampled rows."""
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
    vm.set_attend_balance(True)
    try:
        for call in range(2):
            got = dense.attend(18)
            assert_attention_close(got[0][rows], want_d, f"adaptive dense call {call}")
            got = layer.attend(18, materialized=True)
            assert_attention_close(got[0][rows], want_m, f"adaptive materialized call {call}")
    finally:
        vm.set_attend_balance(False)
