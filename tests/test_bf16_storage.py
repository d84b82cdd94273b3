"""The bf16-storage model of the attention path (tests/bf16_storage.py) against the fp64 oracle,
on the CPU: what error bf16 storage alone admits on the tiny configuration and on the one-token
grid, whose GPU edge test derives its per-call bars from this model.

* Tiny configuration (16 query tokens x 2 heads per call): the model stays within the fixed
  tolerance (max-abs 2e-2, mean-abs 2e-3) on every call of a 6-frame rollout, with room.
* One-token grid (one query row of 32 values per call): the mean error of a single row is a
  noisy statistic, and on some calls bf16 storage alone exceeds the fixed mean-abs 2e-3 and
  relative-L2 1e-2 (3.23e-3 and 1.015e-2 at chunk 5 of batch element 1). No implementation with
  this storage precision can meet the fixed bars there, which is why that test takes the
  model's own error (x1.5) as the bar where it is larger.
* The model itself: with its rounding points it differs from the oracle by a relative L2 well
  under 1e-2, and with the rounding removed it equals the oracle's absorbed form.
"""
import numpy as np

from oracle import videomla_oracle as O
from tests import bf16_storage as S
from workloads import TINY, Dims, make_layer_inputs

GRID1 = Dims(d_model=64, n_heads=1, d_nope=32, d_rope=8, d_c=16, d_v=32, grid_h=1, grid_w=1,
             window_frames=3, chunk_frames=1, rope_pairs=(2, 1, 1))


def _errors(dims, seed, n_frames, batch):
    inp = make_layer_inputs(dims, seed=seed, n_frames=n_frames, batch=batch)
    out = []
    for b in range(batch):
        for fe in range(0, n_frames, dims.chunk_frames):
            want = O.chunk_attention(inp, b, fe)
            got = S.chunk_attention_bf16_storage(inp, b, fe)
            err = np.abs(got - want)
            rel = np.linalg.norm(got - want) / np.linalg.norm(want)
            out.append((b, fe, err.max(), err.mean(), rel))
    return out


def test_tiny_configuration_within_fixed_tolerance():
    for b, fe, mx, mean, rel in _errors(TINY, seed=0, n_frames=6, batch=2):
        assert mx <= 2e-2 and mean <= 1.5e-3 and rel <= 1e-2, (b, fe, mx, mean, rel)


def test_one_token_grid_exceeds_fixed_mean_bar():
    errs = _errors(GRID1, seed=52, n_frames=7, batch=2)
    worst = max(errs, key=lambda e: e[3])
    assert worst[3] > 2e-3, worst            # storage alone exceeds the fixed mean bar
    assert (worst[0], worst[1]) == (1, 5)
    assert abs(worst[3] - 3.228e-3) < 5e-6, worst
    assert worst[4] > 1e-2, worst            # and the relative-L2 bar, on the same call
    assert sum(e[4] > 1e-2 for e in errs) == 1, errs
    assert all(e[2] <= 2e-2 for e in errs), errs


def test_model_without_rounding_is_the_absorbed_form(monkeypatch):
    inp = make_layer_inputs(TINY, seed=3, n_frames=4)
    monkeypatch.setattr(S, "bf16", lambda v: np.asarray(v, dtype=np.float64))
    got = S.chunk_attention_bf16_storage(inp, 0, 3)
    want = O.chunk_attention(inp, 0, 3, absorbed=True)
    assert np.abs(got - want).max() <= 1e-12 * np.abs(want).max()
