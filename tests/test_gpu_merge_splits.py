"""GPU parity of the split merge at every split count it handles in one pass.

out_proj merges the partial results of a row block's key splits (up to four; calls whose row
blocks are split further are merged beforehand by latent_merge). Its loads are laid out per
split count of a wave, one straight-line copy for each of 1, 2, 3 and 4. The headline shape
reaches at most 3 and the tiny shapes at most 2, so this test walks a small shape with the
headline's d_c = 192 through 1..12 workgroups: its first chunk has 4 key tiles per row block
(2 row blocks at batch 2), which gives every largest split count from 1 to 4 under the even
split (the workgroup count is capped at the 8 units). Every output row is compared with the
oracle, under the fixed bars (max-abs 2e-2, mean-abs 2e-3, relative L2 1e-2). The premerged
path is covered by the query-block tests.
"""
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
from workloads import SMALL, make_layer_inputs  # noqa: E402


def _largest_split_count(units_per_row_block, row_blocks, n_wg):
    """The even split's largest number of workgroups sharing one row block: workgroup k takes
    units [floor(k U / G), floor((k + 1) U / G))."""
    T, U = units_per_row_block, units_per_row_block * row_blocks
    G = min(n_wg, U)
    owner = [max(k for k in range(G) if k * U // G <= u) for u in range(U)]
    return max(owner[rb * T + T - 1] - owner[rb * T] + 1 for rb in range(row_blocks))


def test_small_every_split_count(vm):
    d = SMALL
    inp = make_layer_inputs(d, seed=91, n_frames=2, batch=2)
    layer = Layer(vm, inp, packed=True)
    layer.write(0)
    # frames 0..1: 120 keys = 4 tiles of 32 per row block; 240 query rows = one 256-row block
    # per batch element
    tiles = (2 * d.grid_h * d.grid_w + 31) // 32
    seen = set()
    want = [O.chunk_attention(inp, b, 0) for b in range(2)]
    for wg in range(1, 13):
        seen.add(_largest_split_count(tiles, 2, wg))
        got = layer.attend(0, vm.AttendOpts(n_workgroups=wg))
        for b in range(2):
            assert_attention_close(got[b], want[b], f"small wg={wg} b={b}")
    assert seen == {1, 2, 3, 4}, seen
