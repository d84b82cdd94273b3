"""GPU parity of videomla_attend_noalloc (the attention with the library's static scratch array
as its workspace, for callers that cannot allocate) against videomla_attend with a caller-owned
workspace, through the C ABI: two calls in a row, the second on a smaller shape, each bitwise
equal to videomla_attend's output on the same inputs and within the stated tolerance of the
oracle. The array keeps the first call's contents when the second runs."""
import ctypes

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
from tests.gpu_common import Layer, assert_attention_close, bf16_to_f64, host_bits  # noqa: E402
from workloads import SMALL, TINY, make_layer_inputs  # noqa: E402


def _noalloc(vm, layer, fe, out):
    """videomla_attend_noalloc called through the C ABI with raw device pointers."""
    from paper_2605_30351_amd import _lib as L
    d = L.make_dims(layer.inp.dims)
    w = L.VideomlaWindow(fe)
    p = [ctypes.c_void_p(t.data_ptr()) for t in (layer.q_nope, layer.q_r, layer.w_uk, layer.w_uv,
                                                 layer.c_kv, layer.k_r, out)]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return L.raw().videomla_attend_noalloc(ctypes.byref(d), ctypes.byref(w), layer.inp.batch,
                                           *p, stream)


def test_noalloc_matches_attend_on_two_calls(vm):
    cases = ((SMALL, 2, 8, 6, 70), (TINY, 1, 4, 3, 71))  # the second call is the smaller one
    sizes = [vm.attend_workspace_bytes(d, b) for d, b, _, _, _ in cases]
    assert sizes[1] < sizes[0] <= vm.NOALLOC_SCRATCH_BYTES
    for dims, batch, n_frames, fe, seed in cases:
        inp = make_layer_inputs(dims, seed=seed, n_frames=n_frames, batch=batch)
        layer = Layer(vm, inp, packed=True)
        for f in range(0, fe + 1, dims.chunk_frames):
            layer.write(f)
        want = layer.attend(fe).copy()               # videomla_attend, caller's workspace
        out = torch.full_like(layer.out, float("nan"))
        assert _noalloc(vm, layer, fe, out) == 0
        torch.cuda.synchronize()
        got = bf16_to_f64(host_bits(out))
        assert np.array_equal(got, want), f"{dims} batch {batch}: differs from videomla_attend"
        for b in range(batch):
            assert_attention_close(got[b], O.chunk_attention(inp, b, fe),
                                   f"noalloc {dims.d_c}/{dims.n_heads} fe={fe} b={b}")
