"""GPU parity: the HIP path through the C ABI against the fp64 oracle, on the same seeded bf16
inputs.

Bars: cache-write contents equal the oracle rounded to bf16 (nearest-even) for >= 99.9% of
elements, and every element is within one bf16 ulp of it or within 2^-16 of the row's RMS of
it (the fp32 sum over d_model terms carries an absolute error near 1e-7 at unit scale, which
exceeds one ulp only for values within about 2^-16 of zero); slots are bit-exact and every slot
outside the written frames is bitwise unchanged; attention outputs satisfy max-abs <= 2e-2,
mean-abs <= 2e-3 and relative L2 <= 1e-2, the stated tolerance, on every case here except
the peaked-softmax variants.

The peaked variants (queries x4) have outputs of order one, where an absolute 2e-2 is about one
bf16 ulp of the output itself; their bars are scaled by the output magnitude. The path rounds
six times to bf16 (query, latent, RoPE key, probabilities, merged latent, output; unit roundoff
u = 2^-9), and rounding the query and the cached key moves each score by about u|s|, which the
softmax turns into relative weight errors of the same size: max|err| <= max(2e-2, 8u max|out|)
and mean|err| <= max(2e-3, 4u mean|out|), always with the relative-L2 bar.
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
from tests.gpu_common import (Layer, assert_attention_close, check_written_chunk,  # noqa: E402
                              host_bits, sample_rows)
from workloads import TINY, WAN, WAN_PAPER, make_layer_inputs  # noqa: E402


# -------------------------------------------------------------------------------------------
# Tiny configuration: every write, partial and wrapped windows, batch 2, work partitions
# -------------------------------------------------------------------------------------------

@pytest.mark.parametrize("packed", [False, True], ids=["plain_weights", "packed_weights"])
@pytest.mark.parametrize("norm", [True, False])
def test_tiny_rollout_write_and_attend(vm, norm, packed):
    inp = make_layer_inputs(TINY, seed=0, n_frames=6, batch=2, norm=norm)
    layer = Layer(vm, inp, packed=packed)
    exact = total = 0
    for fe in range(6):
        before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
        layer.write(fe)
        for e, n in check_written_chunk(layer, fe, before_c, before_k):
            exact, total = exact + e, total + n
        for wg in (1, 2, 3, 0):
            got = layer.attend(fe, vm.AttendOpts(n_workgroups=wg))
            for b in range(2):
                want = O.chunk_attention(inp, b, fe)
                assert_attention_close(got[b], want, f"tiny fe={fe} b={b} workgroups={wg}")
    assert exact / total >= 0.999, f"{exact}/{total} exactly rounded"


def test_tiny_peaked_softmax(vm):
    inp = make_layer_inputs(TINY, seed=5, n_frames=6, q_gain=4.0)
    layer = Layer(vm, inp)
    for fe in range(6):
        layer.write(fe)
    got = layer.attend(5)
    assert_attention_close(got[0], O.chunk_attention(inp, 0, 5), "tiny peaked", scaled=True)


# -------------------------------------------------------------------------------------------
# Wan2.1-1.3B geometry
# -------------------------------------------------------------------------------------------

def _roll(layer, upto_fe):
    for fe in range(0, upto_fe + 1, layer.inp.dims.chunk_frames):
        layer.write(fe)


@pytest.mark.parametrize("packed", [False, True], ids=["plain_weights", "packed_weights"])
def test_wan_cache_write_evicts_oldest_frames(vm, packed):
    """The 21-frame ring holds frames 0..20; writing frames 21..23 replaces frame slots 0..2
    and leaves the other 18 frames bitwise untouched."""
    inp = make_layer_inputs(WAN, seed=2, n_frames=24)
    layer = Layer(vm, inp, packed=packed)
    _roll(layer, 18)
    before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
    layer.write(21)
    stats = check_written_chunk(layer, 21, before_c, before_k)
    exact = sum(e for e, _ in stats) / sum(n for _, n in stats)
    print(f"wan cache write exactly rounded fraction {exact:.6f}")
    assert exact >= 0.999
    assert np.array_equal(layer.slots.cpu().numpy()[[0, 4679]], [0, 3 * 1560 - 1])


def test_packed_weight_panel_layout(vm):
    """Every 16-byte entry of the packed panel is the documented slice of [W_DKV; W_KR; 0]:
    with OB 16-row blocks per wave slice (2, or 4 beyond 288 outputs), entry
    ((w * nks + k) * OB + ob) * 64 + l holds row 16 OB w + 16 ob + l % 16, columns
    32 k + 8 (l / 16) .. +8 (bitwise, for the tiny, the Wan and the d_c = 512 shapes)."""
    for dims in (TINY, WAN, WAN.replace(d_c=512)):
        inp = make_layer_inputs(dims, seed=3, n_frames=dims.chunk_frames)
        layer = Layer(vm, inp, packed=True)
        torch.cuda.synchronize()
        got = host_bits(layer.w_packed.view(torch.bfloat16)).reshape(-1, 8)
        nks, no = dims.d_model // 32, dims.d_c + dims.d_rope
        OB = 2 if no <= 288 else 4
        nw = (no + 16 * OB - 1) // (16 * OB)
        panel = np.zeros((16 * OB * nw, dims.d_model), np.uint16)
        panel[:dims.d_c], panel[dims.d_c:no] = inp.w_dkv, inp.w_kr
        e = np.arange(nw * nks * OB * 64)
        lane, blk = e % 64, e // 64
        ob, k, w = blk % OB, (blk // OB) % nks, blk // OB // nks
        rows = 16 * OB * w + 16 * ob + lane % 16
        cols = 32 * k + 8 * (lane // 16)
        want = panel[rows[:, None], cols[:, None] + np.arange(8)]
        assert np.array_equal(got, want)


@pytest.mark.parametrize("batch", [2, 3])
def test_wan_batched_packed_write_matches_oracle(vm, batch):
    """Batches whose tokens exceed 32 per compute unit take the wide cache write (one workgroup
    per compute unit, up to 80 tokens: 37 tokens = 3 blocks of 16 at batch 2, 55 = 4 blocks at
    batch 3; blocks span batch elements); the write after a full ring, evicting frames 0..2."""
    inp = make_layer_inputs(WAN, seed=9, n_frames=24, batch=batch)
    layer = Layer(vm, inp, packed=True)
    for fe in range(0, 21, 3):
        layer.write(fe)
    before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
    layer.write(21)
    stats = check_written_chunk(layer, 21, before_c, before_k)
    exact = sum(e for e, _ in stats) / sum(n for _, n in stats)
    assert exact >= 0.999


def test_wan_batch4_packed_write_matches_oracle(vm):
    """Batch 4 (18,720 tokens: the wide cache write, 74 tokens = 5 blocks of 16 per workgroup,
    blocks spanning batch elements)."""
    inp = make_layer_inputs(WAN, seed=8, n_frames=3, batch=4)
    layer = Layer(vm, inp, packed=True)
    before_c, before_k = host_bits(layer.c_kv), host_bits(layer.k_r)
    layer.write(0)
    stats = check_written_chunk(layer, 0, before_c, before_k)
    exact = sum(e for e, _ in stats) / sum(n for _, n in stats)
    assert exact >= 0.999


@pytest.mark.parametrize("variant", ["wan", "peaked", "paper_dims"])
def test_wan_attend_full_window(vm, variant):
    """The wrapped 21-frame window. The measured configuration compares every one of the
    4,680 x 12 output rows with the oracle; the variants compare sampled rows."""
    dims = WAN_PAPER if variant == "paper_dims" else WAN
    inp = make_layer_inputs(dims, seed=1, n_frames=24, q_gain=4.0 if variant == "peaked" else 1.0)
    layer = Layer(vm, inp)
    _roll(layer, 21)
    got = layer.attend(21)
    rows = np.arange(dims.chunk_tokens) if variant == "wan" else sample_rows(dims.chunk_tokens)
    want = O.chunk_attention(inp, 0, 21, rows=rows)
    assert_attention_close(got[0][rows], want, f"wan attend {variant} ({len(rows)} tokens)",
                           scaled=variant == "peaked")


def test_wan_attend_partial_windows_and_work_partitions(vm):
    inp = make_layer_inputs(WAN, seed=6, n_frames=21)
    layer = Layer(vm, inp)
    rows = sample_rows(WAN.chunk_tokens, k=12, seed=1)
    layer.write(0)
    got = layer.attend(0)  # only the chunk itself is in the window
    assert_attention_close(got[0][rows], O.chunk_attention(inp, 0, 0, rows=rows), "wan fe=0")
    for fe in range(3, 19, 3):
        layer.write(fe)
    want = O.chunk_attention(inp, 0, 18, rows=rows)  # exactly 21 frames, no wrap yet
    for wg in (0, 1, 37, 300):
        got = layer.attend(18, vm.AttendOpts(n_workgroups=wg))
        assert_attention_close(got[0][rows], want, f"wan fe=18 workgroups={wg}")


def test_wan_attend_is_deterministic(vm):
    """Two calls give bitwise identical outputs in the default (even) partition and in the
    frozen partition the benchmark measures (weights calibrated by adaptive calls on the same
    workspace, then frozen); the frozen outputs match the oracle."""
    inp = make_layer_inputs(WAN, seed=7, n_frames=24)
    layer = Layer(vm, inp)
    _roll(layer, 21)
    a = layer.attend(21).copy()
    b = layer.attend(21)
    assert np.array_equal(a, b)
    ws = torch.empty(vm.attend_workspace_bytes(WAN, 1), dtype=torch.uint8, device="cuda")
    for _ in range(3):
        layer.attend(21, vm.AttendOpts(partition="adaptive"), ws=ws)
    frozen = vm.AttendOpts(partition="frozen")
    fa = layer.attend(21, frozen, ws=ws).copy()
    fb = layer.attend(21, frozen, ws=ws)
    assert np.array_equal(fa, fb)
    rows = sample_rows(WAN.chunk_tokens, k=12, seed=7)
    assert_attention_close(fa[0][rows], O.chunk_attention(inp, 0, 21, rows=rows), "wan frozen")
    assert_attention_close(fa[0], a[0], "frozen vs even split")
