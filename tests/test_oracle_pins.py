"""Pins of the fp64 oracle against things other than itself: values the paper prints, a case
worked by hand, closed forms, invariants the paper relies on, library routines and brute force.

Each test names the mistake it is there to catch.
"""
import collections
import dataclasses
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import videomla_oracle as O
from workloads import TINY, WAN, WAN_PAPER, Dims, bf16_bits_to_f32, f32_to_bf16_bits, make_layer_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ------------------------------------------------------------------------------------------
# bf16 rounding
# ------------------------------------------------------------------------------------------

def test_bf16_round_matches_torch_on_fp32_values():
    """Catches a wrong rounding mode (truncation, ties-away) in the oracle's RNE."""
    rng = np.random.default_rng(0)
    v = rng.standard_normal(200000).astype(np.float32) * np.float32(3.0)
    # exact ties: bf16 value plus half an ulp
    base = bf16_bits_to_f32(f32_to_bf16_bits(v[:1000]))
    ties = (base + np.float32(0.5) * np.exp2(np.floor(np.log2(np.abs(base)))) * np.float32(2.0 ** -7)).astype(np.float32)
    v = np.concatenate([v, ties, -ties, np.float32([0.0, 1.0, -2.5, 1e-30, 3e-39])])
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = O.round_to_bf16_bits(v.astype(np.float64))
    assert np.array_equal(got, want)


def test_bf16_round_brute_force_on_fp64_values():
    """Catches double rounding (fp64 -> fp32 -> bf16) in the direct fp64 -> bf16 rounding."""
    rng = np.random.default_rng(1)
    v = rng.standard_normal(3000) * 10.0
    got = O.round_to_bf16_bits(v)
    for val, g in zip(v, got):
        lo = int(f32_to_bf16_bits(np.float32([val]))[0])
        cands = {lo - 1, lo, lo + 1}
        best = min(cands, key=lambda b: (abs(float(bf16_bits_to_f32(np.uint16([b]))[0]) - val), b & 1))
        assert g == best


# ------------------------------------------------------------------------------------------
# Memory arithmetic printed in the paper
# ------------------------------------------------------------------------------------------

def test_memory_figures_printed_in_paper():
    """Catches a wrong per-token cache formula (e.g. counting k^R per head)."""
    g = _golden("paper_memory_figures.json")
    latent, dense = O.cache_scalars_per_token(WAN), O.dense_scalars_per_token(WAN)
    assert latent == g["cache_scalars_per_token"]["value"]
    assert dense == g["dense_scalars_per_token"]["value"]
    assert round(100 * (1 - latent / dense), 1) == g["reduction_percent"]["value"]
    assert round(dense / latent, 1) == g["reduction_factor"]["value"]
    for dc, want in zip(g["table5_mem_ratio"]["d_c"], g["table5_mem_ratio"]["value"]):
        assert round(dense / O.cache_scalars_per_token(WAN.replace(d_c=dc)), 2) == want
    d = g["dense_cache_scalars_billion"]
    scalars = d["frames"] * d["tokens_per_frame"] * d["layers"] * dense
    assert round(scalars / 1e9, 2) == d["value"]
    assert round(scalars * 2 / 1e9, 1) == g["dense_cache_gb_bf16"]["value"]
    scd = g["scd_reduction_percent"]["cached_layers"]
    assert round(100 * (1 - scd / d["layers"]), 1) == g["scd_reduction_percent"]["value"]
    assert round(scd * dense / (d["layers"] * latent), 1) == g["vs_scd_factor"]["value"]
    # the paper-dims variant caches the same 224 scalars
    assert O.cache_scalars_per_token(WAN_PAPER) == latent


# ------------------------------------------------------------------------------------------
# The two-token case worked by hand
# ------------------------------------------------------------------------------------------

HAND = Dims(d_model=2, n_heads=1, d_nope=2, d_rope=2, d_c=2, d_v=2, grid_h=1, grid_w=1,
            window_frames=2, chunk_frames=1, rope_pairs=(1, 0, 0), rope_base=10000.0)


def _hand_attend(shift, fn):
    q_nope = np.array([[[1.0, 0.0]]])
    q_r = np.array([[[1.0, 0.0]]])
    c = np.array([[1.0, 0.0], [0.0, 1.0]])
    kr = np.array([[1.0, 0.0], [1.0, 0.0]])
    t_k = np.array([0, 1]) + shift
    k_rope = O.rope3d(kr, t_k, np.zeros(2), np.zeros(2), HAND)
    q_rope = O.rope3d(q_r, np.array([1 + shift]), np.zeros(1), np.zeros(1), HAND)
    eye = np.eye(2)
    return fn(q_nope, q_rope, eye, eye, c, k_rope, HAND), q_rope, k_rope


@pytest.mark.parametrize("absorbed", [False, True])
def test_two_token_hand_case(absorbed):
    """Catches a dropped RoPE or NoPE score term, a wrong scale, or a wrong softmax/value sum."""
    g = _golden("two_token_hand_case.json")
    fn = O.attend_absorbed if absorbed else O.attend_unabsorbed
    o, q_rope, k_rope = _hand_attend(0, fn)
    s = np.array([(1.0 + q_rope[0, 0] @ k_rope[0]) / 2, (0.0 + q_rope[0, 0] @ k_rope[1]) / 2])
    np.testing.assert_allclose(s, g["scores"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(o[0, 0], g["out"], rtol=0, atol=1e-15)
    o_shift, _, _ = _hand_attend(g["shift_t"], fn)
    np.testing.assert_allclose(o_shift[0, 0], g["out"], rtol=0, atol=1e-14)


# ------------------------------------------------------------------------------------------
# RoPE
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("dims", [TINY, WAN, WAN_PAPER])
def test_rope_single_axis_is_complex_multiplication(dims):
    """Catches a wrong rotation direction, half-split instead of interleaved pairs, a wrong
    frequency exponent, or an axis rotated by another axis' coordinate."""
    rng = np.random.default_rng(2)
    v = rng.standard_normal((5, dims.d_rope))
    layout = O.rope_axis_layout(dims)
    for axis in range(3):
        pos = [np.zeros(5), np.zeros(5), np.zeros(5)]
        pos[axis] = np.array([0, 1, 3, 17, 239], dtype=float)
        got = O.rope3d(v, *pos, dims)
        want = v.copy()
        start, npairs, band = layout[axis]
        for k in range(npairs):
            z = v[:, start + 2 * k] + 1j * v[:, start + 2 * k + 1]
            z = z * np.exp(1j * pos[axis] * dims.rope_base ** (-(2.0 * k) / band))
            want[:, start + 2 * k] = z.real
            want[:, start + 2 * k + 1] = z.imag
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-13)


def test_rope_axis_split_matches_dims():
    assert [(s, n) for s, n, _ in O.rope_axis_layout(WAN)] == [(0, 8), (16, 4), (24, 4)]
    assert [(s, n) for s, n, _ in O.rope_axis_layout(WAN_PAPER)] == [(0, 6), (12, 5), (22, 5)]
    assert [(s, n) for s, n, _ in O.rope_axis_layout(TINY)] == [(0, 2), (4, 1), (6, 1)]
    assert [b for _, _, b in O.rope_axis_layout(WAN_PAPER)] == [44, 42, 42]


@pytest.mark.parametrize("dims", [TINY, WAN_PAPER])
def test_rope_scores_depend_only_on_relative_position(dims):
    """The property the paper's window re-indexing relies on: shifting every (t, h, w) of
    queries and keys by one offset leaves all q_rope.k_rope scores unchanged. Catches queries
    and keys rotated with different conventions."""
    rng = np.random.default_rng(3)
    q = rng.standard_normal((7, dims.d_rope))
    k = rng.standard_normal((9, dims.d_rope))
    pq = [rng.integers(0, 40, 7), rng.integers(0, 30, 7), rng.integers(0, 52, 7)]
    pk = [rng.integers(0, 40, 9), rng.integers(0, 30, 9), rng.integers(0, 52, 9)]
    s0 = O.rope3d(q, *pq, dims) @ O.rope3d(k, *pk, dims).T
    for off in [(5, 0, 0), (0, -3, 7), (200, 11, -13)]:
        s1 = O.rope3d(q, *[p + o for p, o in zip(pq, off)], dims) @ \
            O.rope3d(k, *[p + o for p, o in zip(pk, off)], dims).T
        np.testing.assert_allclose(s1, s0, rtol=0, atol=1e-12)
    # and a relative offset does change them
    s2 = O.rope3d(q, pq[0] + 1, pq[1], pq[2], dims) @ O.rope3d(k, *pk, dims).T
    assert np.max(np.abs(s2 - s0)) > 1e-3


def test_rope_zero_position_is_identity_and_norm_preserving():
    rng = np.random.default_rng(4)
    v = rng.standard_normal((3, WAN.d_rope))
    np.testing.assert_array_equal(O.rope3d(v, np.zeros(3), np.zeros(3), np.zeros(3), WAN), v)
    r = O.rope3d(v, np.array([3, 9, 23]), np.array([1, 5, 29]), np.array([0, 51, 7]), WAN)
    pair_norm = lambda a: a[:, 0::2] ** 2 + a[:, 1::2] ** 2
    np.testing.assert_allclose(pair_norm(r), pair_norm(v), rtol=1e-13)


# ------------------------------------------------------------------------------------------
# Slot map and window
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("W_f,chunk,grid", [(3, 1, (4, 4)), (21, 3, (2, 3)), (7, 3, (1, 2)), (5, 2, (3, 1))])
def test_slot_map_matches_fifo_simulation(W_f, chunk, grid):
    """Brute force: a FIFO of frames (deque) holding the most recent W_f frames must contain
    exactly the frames the closed-form slot map places in the ring, every cached token has a
    distinct slot, and the attended window is the chunk plus the newest past frames."""
    dims = Dims(d_model=8, n_heads=1, d_nope=2, d_rope=2, d_c=2, d_v=2, grid_h=grid[0],
                grid_w=grid[1], window_frames=W_f, chunk_frames=chunk, rope_pairs=(1, 0, 0))
    fifo = collections.deque(maxlen=W_f)
    ring_frame = {}  # slot -> (f, y, x)
    for frame_end in range(0, 6 * W_f, chunk):
        n = np.arange(dims.chunk_tokens)
        f, y, x = O.token_position(n, frame_end, dims)
        slots = O.ring_slot(f, y, x, dims)
        assert len(set(slots.tolist())) == len(slots)
        for s, ff, yy, xx in zip(slots, f, y, x):
            ring_frame[int(s)] = (int(ff), int(yy), int(xx))
        for ff in range(frame_end, frame_end + chunk):
            fifo.append(ff)
        held = sorted({v[0] for v in ring_frame.values()})
        assert held == sorted(fifo)
        lo, hi = O.window_frame_range(frame_end, dims)
        assert list(range(lo, hi)) == sorted(fifo)
        assert sorted(O.ring_after_writes(hi, dims)[O.ring_after_writes(hi, dims) >= 0].tolist()) == sorted(fifo)
        # every held token sits in its own slot, row-major inside its frame slot
        for s, (ff, yy, xx) in ring_frame.items():
            assert s == (ff % W_f) * dims.hw + yy * dims.grid_w + xx
        assert all(0 <= s < dims.window_tokens for s in ring_frame)


# ------------------------------------------------------------------------------------------
# Compress and RMSNorm
# ------------------------------------------------------------------------------------------

def test_compress_one_hot_input_picks_a_column():
    """Catches a transposed W_DKV / W_KR (the paper stores W_down^KV as d_c x d)."""
    rng = np.random.default_rng(5)
    w_dkv = rng.standard_normal((TINY.d_c, TINY.d_model))
    w_kr = rng.standard_normal((TINY.d_rope, TINY.d_model))
    x = np.zeros((3, TINY.d_model))
    x[0, 5] = 1.0; x[1, 63] = 2.0; x[2, 0] = -1.0
    c, kr = O.compress(x, w_dkv, w_kr, None, TINY)
    np.testing.assert_array_equal(c, np.stack([w_dkv[:, 5], 2 * w_dkv[:, 63], -w_dkv[:, 0]]))
    np.testing.assert_array_equal(kr, np.stack([w_kr[:, 5], 2 * w_kr[:, 63], -w_kr[:, 0]]))


def test_rmsnorm_closed_forms():
    """With unit gain the normalized latent has mean square 1/(1+eps/ms); scaling the input
    leaves it unchanged (up to eps); a gain multiplies channels. Catches a missing mean or
    sqrt, or the gain applied before the norm."""
    rng = np.random.default_rng(6)
    x = rng.standard_normal((4, TINY.d_model))
    w = rng.standard_normal((TINY.d_c, TINY.d_model))
    wk = rng.standard_normal((TINY.d_rope, TINY.d_model))
    d0 = TINY.replace(kv_norm_eps=0.0)
    c, _ = O.compress(x, w, wk, np.ones(TINY.d_c), d0)
    np.testing.assert_allclose(np.mean(c * c, axis=1), 1.0, rtol=1e-14)
    c2, _ = O.compress(7.5 * x, w, wk, np.ones(TINY.d_c), d0)
    np.testing.assert_allclose(c2, c, rtol=1e-13)
    g = np.arange(1, TINY.d_c + 1, dtype=float)
    c3, _ = O.compress(x, w, wk, g, d0)
    np.testing.assert_allclose(c3, c * g, rtol=1e-14)
    raw, _ = O.compress(x, w, wk, None, d0)
    eps = 1e-6
    c4, _ = O.compress(x, w, wk, np.ones(TINY.d_c), TINY.replace(kv_norm_eps=eps))
    ms = np.mean(raw * raw, axis=1, keepdims=True)
    np.testing.assert_allclose(c4, raw / np.sqrt(ms + eps), rtol=1e-14)


# ------------------------------------------------------------------------------------------
# Attention: absorbed vs reconstructed, library routine, closed forms, head indexing
# ------------------------------------------------------------------------------------------

def _rand_attn(dims, nq, S, seed):
    rng = np.random.default_rng(seed)
    q_nope = rng.standard_normal((nq, dims.n_heads, dims.d_nope))
    q_rope = rng.standard_normal((nq, dims.n_heads, dims.d_rope))
    w_uk = rng.standard_normal((dims.n_heads * dims.d_nope, dims.d_c)) / np.sqrt(dims.d_c)
    w_uv = rng.standard_normal((dims.n_heads * dims.d_v, dims.d_c)) / np.sqrt(dims.d_c)
    c = rng.standard_normal((S, dims.d_c))
    kr = rng.standard_normal((S, dims.d_rope))
    return q_nope, q_rope, w_uk, w_uv, c, kr


@pytest.mark.parametrize("dims,nq,S", [(TINY, 16, 48), (WAN, 20, 300), (WAN_PAPER, 9, 130)])
def test_absorbed_equals_reconstructed(dims, nq, S):
    """Eqs. 8-11: absorbing W_UK into the query and applying W_UV after the latent sum is the
    same computation. Catches a transposed up-projection or a wrong head slice in either."""
    args = _rand_attn(dims, nq, S, 7)
    a = O.attend_unabsorbed(*args, dims)
    b = O.attend_absorbed(*args, dims)
    assert np.max(np.abs(a - b)) <= 1e-12 * max(1.0, np.max(np.abs(a)))


def test_attention_core_matches_library_sdpa():
    """At zero positions RoPE is the identity, so the oracle must equal the library's scaled
    dot-product attention over K = [c W_UK_h^T | k^R], V = c W_UV_h^T (fp64, CPU)."""
    dims = WAN
    q_nope, q_r, w_uk, w_uv, c, kr = _rand_attn(dims, 11, 257, 8)
    zero = np.zeros(257)
    kro = O.rope3d(kr, zero, zero, zero, dims)
    qro = O.rope3d(q_r, np.zeros(11), np.zeros(11), np.zeros(11), dims)
    got = O.attend_unabsorbed(q_nope, qro, w_uk, w_uv, c, kro, dims, row_block=4)
    for h in range(dims.n_heads):
        K = torch.from_numpy(np.concatenate([c @ w_uk[h * 128:(h + 1) * 128].T, kr], 1))
        V = torch.from_numpy(c @ w_uv[h * 128:(h + 1) * 128].T)
        Q = torch.from_numpy(np.concatenate([q_nope[:, h], q_r[:, h]], 1))
        want = torch.nn.functional.scaled_dot_product_attention(
            Q[None], K[None], V[None], scale=1 / math.sqrt(160)).numpy()[0]
        np.testing.assert_allclose(got[:, h], want, rtol=1e-12, atol=1e-14)


def test_identical_keys_give_the_value_exactly():
    """Closed form: if every window token carries the same latents the softmax is uniform and
    o_h = W_UV_h c for any query."""
    dims = TINY
    q_nope, q_rope, w_uk, w_uv, c, kr = _rand_attn(dims, 5, 48, 9)
    c[:] = c[0]
    kr[:] = kr[0]
    o = O.attend_unabsorbed(q_nope, q_rope, w_uk, w_uv, c, kr, dims)
    for h in range(dims.n_heads):
        np.testing.assert_allclose(o[:, h], np.broadcast_to(w_uv[h * 32:(h + 1) * 32] @ c[0], (5, 32)),
                                   rtol=1e-13, atol=1e-15)


def test_dominant_key_limit():
    """Closed form: with one key far ahead in score the output tends to that key's value."""
    dims = TINY
    q_nope, q_rope, w_uk, w_uv, c, kr = _rand_attn(dims, 3, 48, 10)
    q_nope[:] = 0.0
    kr[:] = 0.0
    kr[17] = 1.0
    q_rope[:] = 400.0
    o = O.attend_unabsorbed(q_nope, q_rope, w_uk, w_uv, c, kr, dims)
    for h in range(dims.n_heads):
        np.testing.assert_allclose(o[:, h], np.broadcast_to(w_uv[h * 32:(h + 1) * 32] @ c[17], (3, 32)),
                                   rtol=1e-12, atol=1e-12)


def test_head_permutation_equivariance():
    """Permuting heads in the queries and in the row blocks of W_UK / W_UV permutes the output
    heads. Catches the query of head h scored against another head's key projection."""
    dims = WAN_PAPER
    q_nope, q_rope, w_uk, w_uv, c, kr = _rand_attn(dims, 6, 90, 11)
    perm = np.array([3, 0, 11, 1, 2, 10, 4, 9, 5, 8, 6, 7])
    rows = lambda w, d: np.concatenate([w[h * d:(h + 1) * d] for h in perm])
    a = O.attend_unabsorbed(q_nope, q_rope, w_uk, w_uv, c, kr, dims)
    b = O.attend_unabsorbed(q_nope[:, perm], q_rope[:, perm], rows(w_uk, dims.d_nope),
                            rows(w_uv, dims.d_v), c, kr, dims)
    np.testing.assert_allclose(b, a[:, perm], rtol=1e-13, atol=1e-15)
    # and heads do differ from each other
    assert np.max(np.abs(a[:, 0] - a[:, 1])) > 1e-3


def test_row_blocking_does_not_change_results():
    dims = TINY
    args = _rand_attn(dims, 16, 48, 12)
    np.testing.assert_allclose(O.attend_unabsorbed(*args, dims, row_block=3),
                               O.attend_unabsorbed(*args, dims, row_block=512), rtol=0, atol=1e-14)


# ------------------------------------------------------------------------------------------
# End to end: window-relative rotation (the paper's) equals rotation at absolute positions
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("frame_end", [0, 1, 5])
def test_rotate_at_read_window_relative_equals_absolute(frame_end):
    """Without a sink frame, the paper's window-relative re-indexing is one uniform temporal
    shift of every query and key, so attention results are unchanged."""
    inp = make_layer_inputs(TINY, seed=0, n_frames=6)
    a = O.chunk_attention(inp, 0, frame_end)
    lo, _ = O.window_frame_range(frame_end, TINY)
    b = O.chunk_attention(inp, 0, frame_end, rotate_origin=lo)
    c = O.chunk_attention(inp, 0, frame_end, absorbed=True)
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-12)
    np.testing.assert_allclose(c, a, rtol=0, atol=1e-12)


def test_window_partial_at_rollout_start():
    assert O.window_frame_range(0, TINY) == (0, 1)
    assert O.window_frame_range(1, TINY) == (0, 2)
    assert O.window_frame_range(5, TINY) == (3, 6)
    assert O.window_frame_range(21, WAN) == (3, 24)
    assert O.window_frame_range(0, WAN) == (0, 3)


def test_cache_write_positions_and_slots():
    """Chunk tokens are frames in order, row-major over the grid; the written slot of token n
    at frame_end=21 (Wan geometry) is the slot of frame (21 + n // 1560) mod 21."""
    n = np.array([0, 51, 52, 1559, 1560, 4679])
    f, y, x = O.token_position(n, 21, WAN)
    assert f.tolist() == [21, 21, 21, 21, 22, 23]
    assert y.tolist() == [0, 0, 1, 29, 0, 29]
    assert x.tolist() == [0, 51, 0, 51, 0, 51]
    assert O.ring_slot(f, y, x, WAN).tolist() == [0, 51, 52, 1559, 1560, 2 * 1560 + 1559]


# ------------------------------------------------------------------------------------------
# Dense per-head comparator
# ------------------------------------------------------------------------------------------

def test_dense_head_rope_split():
    """The full-head split rule gives (44, 42, 42) channels at d = 128, Wan's own axis groups,
    and (12, 10, 10) channels = (6, 5, 5) pairs at d = 32, the paper's RoPE-key split."""
    hd = O.dense_head_rope_dims(WAN)
    assert hd.d_rope == 128 and hd.rope_pairs == (22, 21, 21) and hd.rope_band_dim == (44, 42, 42)
    hd32 = O.dense_head_rope_dims(WAN.replace(d_v=32))
    assert hd32.rope_pairs == WAN_PAPER.rope_pairs


def test_dense_zero_positions_equal_sdpa():
    """At position 0 every rotation is the identity, so the comparator is plain scaled
    dot-product attention per head (library routine, fp64)."""
    rng = np.random.default_rng(11)
    dims = TINY
    nq, S, H, d = 9, 23, dims.n_heads, dims.d_v
    q, k, v = rng.standard_normal((nq, H, d)), rng.standard_normal((S, H, d)), rng.standard_normal((S, H, d))
    zero = (np.zeros(nq, np.int64),) * 3
    got = O.dense_attend(q, k, v, zero, dims)
    for h in range(H):
        want = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[:, h])[None], torch.from_numpy(k[:, h])[None],
            torch.from_numpy(v[:, h])[None]).numpy()[0]
        np.testing.assert_allclose(got[:, h], want, rtol=0, atol=1e-12)


def test_dense_equals_latent_with_composed_weights():
    """With W_K,h = W_UK,h W_DKV and W_V,h = W_UV,h W_DKV (no norm, no RoPE key, no rotation),
    dense per-head attention and the latent reconstruction of Eq. 2 compute the same thing:
    the latent cache is a factorization of the dense one."""
    dims = TINY.replace(softmax_scale=1.0 / math.sqrt(TINY.d_nope + TINY.d_rope))
    assert dims.d_nope == dims.d_v
    rng = np.random.default_rng(12)
    H, dn, dc, dv, D = dims.n_heads, dims.d_nope, dims.d_c, dims.d_v, dims.d_model
    x = rng.standard_normal((40, D))
    w_dkv, w_uk, w_uv = rng.standard_normal((dc, D)), rng.standard_normal((H * dn, dc)), rng.standard_normal((H * dv, dc))
    c = x @ w_dkv.T
    q = rng.standard_normal((7, H, dn))
    latent = O.attend_unabsorbed(q, np.zeros((7, H, dims.d_rope)), w_uk, w_uv, c,
                                 np.zeros((40, dims.d_rope)), dims)
    w_k = np.concatenate([w_uk[h * dn:(h + 1) * dn] @ w_dkv for h in range(H)])
    w_v = np.concatenate([w_uv[h * dv:(h + 1) * dv] @ w_dkv for h in range(H)])
    k = (x @ w_k.T).reshape(40, H, dv)
    v = (x @ w_v.T).reshape(40, H, dv)
    dense = O.dense_attend(q, k, v, (np.zeros(7, np.int64),) * 3, dims)
    np.testing.assert_allclose(dense, latent, rtol=1e-11, atol=1e-11)


def test_dense_scores_invariant_under_common_shift():
    """Shifting every query and key position by the same (t, h, w) offset leaves the comparator's
    output unchanged (relative-position property of the full-head RoPE)."""
    dims = TINY
    rng = np.random.default_rng(13)
    x = rng.standard_normal((20, dims.d_model))
    w_k = rng.standard_normal((dims.n_heads * dims.d_v, dims.d_model)) / 8
    w_v = rng.standard_normal((dims.n_heads * dims.d_v, dims.d_model)) / 8
    q = rng.standard_normal((5, dims.n_heads, dims.d_v))
    kpos = (rng.integers(0, 9, 20), rng.integers(0, 4, 20), rng.integers(0, 4, 20))
    qpos = (rng.integers(0, 9, 5), rng.integers(0, 4, 5), rng.integers(0, 4, 5))
    shift = (17, 3, -5)
    k, v = O.dense_kv(x, w_k, w_v, kpos, dims)
    ks, _ = O.dense_kv(x, w_k, w_v, tuple(p + s for p, s in zip(kpos, shift)), dims)
    a = O.dense_attend(q, k, v, qpos, dims)
    b = O.dense_attend(q, ks, v, tuple(p + s for p, s in zip(qpos, shift)), dims)
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-11)


def test_dense_cache_write_places_like_the_latent_cache():
    from workloads import make_dense_inputs
    inp = make_dense_inputs(TINY, seed=3, n_frames=6)
    hw = TINY.hw
    got = O.dense_cache_write(inp.x[0, 5 * hw:6 * hw], inp.w_k, inp.w_v, 5, TINY)
    f, y, x = O.token_position(np.arange(hw), 5, TINY)
    assert np.array_equal(got["slots"], O.ring_slot(f, y, x, TINY))
    assert got["k"].shape == (hw, TINY.n_heads, TINY.d_v)


# ------------------------------------------------------------------------------------------
# Sink frame + local window with window-relative RoPE re-indexing
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("W_f,S,chunk,grid", [(4, 1, 1, (2, 2)), (7, 1, 3, (1, 3)), (9, 2, 3, (2, 1))])
def test_sink_slot_map_matches_simulation(W_f, S, chunk, grid):
    """Brute force: the first S frames stay in the cache for good and a FIFO (deque) of the
    most recent W_f - S later frames holds the rest. The closed-form slot map must hold exactly
    those frames, the context of each chunk must be them in time order, and slots are distinct."""
    dims = Dims(d_model=8, n_heads=1, d_nope=2, d_rope=2, d_c=2, d_v=2, grid_h=grid[0],
                grid_w=grid[1], window_frames=W_f, chunk_frames=chunk, rope_pairs=(1, 0, 0),
                sink_frames=S)
    sink, fifo = [], collections.deque(maxlen=W_f - S)
    ring_frame = {}
    for frame_end in range(0, 8 * W_f, chunk):
        n = np.arange(dims.chunk_tokens)
        f, y, x = O.token_position(n, frame_end, dims)
        slots = O.ring_slot(f, y, x, dims)
        assert len(set(slots.tolist())) == len(slots)
        for s, ff, yy, xx in zip(slots, f, y, x):
            ring_frame[int(s)] = (int(ff), int(yy), int(xx))
        for ff in range(frame_end, frame_end + chunk):
            (sink if ff < S else fifo).append(ff)
        held = sorted({v[0] for v in ring_frame.values()})
        assert held == sorted(sink + list(fifo))
        assert O.context_frames(frame_end, dims) == sink + list(fifo)
        rw = O.ring_after_writes(frame_end + chunk, dims)
        assert sorted(rw[rw >= 0].tolist()) == held
        assert all(0 <= s < dims.window_tokens for s in ring_frame)
        # the sink frames never move
        for ff in sink:
            assert int(O.frame_slot(ff, dims)) == ff


def test_sink_local_time_table():
    """The paper's long-rollout context (one sink frame, six recent frames, 3-frame chunks):
    the sink takes local time 0 and the recent frames 1..6 however far the rollout has gone;
    before the cache is full local time is the absolute frame index."""
    from workloads import WAN_SINK
    assert O.context_frames(0, WAN_SINK) == [0, 1, 2]
    assert O.context_frames(3, WAN_SINK) == [0, 1, 2, 3, 4, 5]
    assert O.context_frames(6, WAN_SINK) == [0, 3, 4, 5, 6, 7, 8]
    assert O.context_frames(237, WAN_SINK) == [0, 234, 235, 236, 237, 238, 239]
    assert O.local_time([0, 1, 2], 0, WAN_SINK).tolist() == [0, 1, 2]
    assert O.local_time([0, 3, 5], 3, WAN_SINK).tolist() == [0, 3, 5]
    assert O.local_time([0, 3, 6, 8], 6, WAN_SINK).tolist() == [0, 1, 4, 6]
    assert O.local_time([0, 234, 237, 239], 237, WAN_SINK).tolist() == [0, 1, 4, 6]
    # frame slots: the sink keeps slot 0, frames 1.. cycle through slots 1..6
    assert O.frame_slot([0, 1, 6, 7, 12, 239], WAN_SINK).tolist() == [0, 1, 6, 1, 6, 5]


def test_sink_equals_plain_window_before_eviction():
    """While every generated frame still fits in the cache, the sink context is the plain
    window, local time is absolute time, and both modes give the same attention."""
    from workloads import TINY_SINK
    plain = TINY_SINK.replace(sink_frames=0)
    inp_s = make_layer_inputs(TINY_SINK, seed=3, n_frames=4)
    inp_p = make_layer_inputs(plain, seed=3, n_frames=4)
    for frame_end in range(4):
        a = O.chunk_attention(inp_s, 0, frame_end)
        b = O.chunk_attention(inp_p, 0, frame_end)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def _absolute_time_attention(inp, frame_end):
    """The same context keys and queries rotated at absolute time instead of window-local
    time (what the cache would give if the re-indexing were skipped)."""
    d = inp.dims
    frames = O.context_frames(frame_end, d)
    x = O.bf16_bits_to_f64(np.concatenate([inp.x[0][f * d.hw:(f + 1) * d.hw] for f in frames]))
    c, kr = O.compress(x, O.bf16_bits_to_f64(inp.w_dkv), O.bf16_bits_to_f64(inp.w_kr),
                       O.bf16_bits_to_f64(inp.gamma), d)
    n = np.arange(x.shape[0])
    f = np.asarray(frames)[n // d.hw]
    k = O.rope3d(kr, f, (n % d.hw) // d.grid_w, n % d.grid_w, d)
    rows = np.arange(d.chunk_tokens)
    q_rope = O.query_rope(O.bf16_bits_to_f64(inp.q_r[0]), O.token_position(rows, frame_end, d), d)
    return O.attend_unabsorbed(O.bf16_bits_to_f64(inp.q_nope[0]), q_rope,
                               O.bf16_bits_to_f64(inp.w_uk), O.bf16_bits_to_f64(inp.w_uv), c, k, d)


def test_sink_rollout_depends_only_on_window_content():
    """Window-relative re-indexing: two chunks far apart in the rollout whose contexts hold the
    same content (same sink frame, same recent frames) give the same attention, so positions
    stay bounded. Rotating at absolute time instead gives different results (the sink's offset
    to the queries grows), which shows this check can fail."""
    from workloads import TINY_SINK
    d = TINY_SINK
    inp = make_layer_inputs(d, seed=4, n_frames=40)
    x = inp.x.copy()
    F1, F2 = 5, 37
    for k in range(d.window_frames - d.sink_frames):   # recent frames of F2 := those of F1
        a, b = F1 - k, F2 - k
        x[:, b * d.hw:(b + 1) * d.hw] = x[:, a * d.hw:(a + 1) * d.hw]
    inp = dataclasses.replace(inp, x=x)
    o1 = O.chunk_attention(inp, 0, F1)
    o2 = O.chunk_attention(inp, 0, F2)
    np.testing.assert_allclose(o2, o1, rtol=0, atol=1e-12)
    assert np.abs(_absolute_time_attention(inp, F2) - o2).max() > 1e-4


def test_sink_cache_write_keeps_keys_unrotated():
    """With a sink the cache holds the position-free key W_R^K x; without one it holds the key
    rotated at the token's absolute position."""
    from workloads import TINY_SINK
    inp = make_layer_inputs(TINY_SINK, seed=5, n_frames=8)
    fe = 6
    xs = inp.x[0][fe * TINY_SINK.hw:(fe + 1) * TINY_SINK.hw]
    ref = O.cache_write(xs, inp.w_dkv, inp.w_kr, inp.gamma, fe, TINY_SINK)
    kr = O.bf16_bits_to_f64(xs) @ O.bf16_bits_to_f64(inp.w_kr).T
    np.testing.assert_allclose(ref["k_cached"], kr, rtol=0, atol=1e-12)
    # frame 6 lives in frame slot 1 + (6 - 1) mod 3 = 3
    assert (ref["slots"] // TINY_SINK.hw == 3).all()
    plain = O.cache_write(xs, inp.w_dkv, inp.w_kr, inp.gamma, fe, TINY_SINK.replace(sink_frames=0))
    f, y, x = O.token_position(np.arange(TINY_SINK.hw), fe, TINY_SINK)
    np.testing.assert_allclose(plain["k_cached"], O.rope3d(kr, f, y, x, TINY_SINK), rtol=0, atol=1e-12)


# ------------------------------------------------------------------------------------------
# Whole attention layer (query path + output projection)
# ------------------------------------------------------------------------------------------

def _full_tiny(sink=False, seed=10, n_frames=6, d_q=48):
    from workloads import TINY_SINK, make_full_layer_inputs
    return make_full_layer_inputs(TINY_SINK if sink else TINY, seed=seed, n_frames=n_frames, d_q=d_q)


@pytest.mark.parametrize("sink", [False, True])
@pytest.mark.parametrize("frame_end", [0, 2, 5])
def test_layer_absorbed_equals_reconstructed(sink, frame_end):
    """Eqs. 8-11: the latent form with A_h = (W_up,h^Q)^T W_up,h^K and B_h = W_h^O W_up,h^V
    equals the reconstructed per-head form followed by W_O."""
    inp = _full_tiny(sink)
    a = O.attention_layer(inp, 0, frame_end)
    b = O.attention_layer_absorbed(inp, 0, frame_end)
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-12 * np.abs(a).max())


def test_layer_query_latent_is_normalized(monkeypatch):
    """With the positional queries zeroed, the scores see only normalized latents, so scaling
    every activation by a constant leaves the layer output unchanged (up to eps). A planted
    mistake, c^Q without its RMSNorm, breaks the invariance."""
    inp = _full_tiny()
    inp = dataclasses.replace(inp, w_qr=np.zeros_like(inp.w_qr))
    x4 = f32_to_bf16_bits(bf16_bits_to_f32(inp.x) * np.float32(4.0))  # exact in bf16
    a = O.attention_layer(inp, 0, 3)
    b = O.attention_layer(dataclasses.replace(inp, x=x4), 0, 3)
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-5 * np.abs(a).max())
    monkeypatch.setattr(O, "query_latent", lambda x, w_dq, gamma_q, dims: gamma_q * (x @ w_dq.T))
    a2 = O.attention_layer(inp, 0, 3)
    b2 = O.attention_layer(dataclasses.replace(inp, x=x4), 0, 3)
    assert np.abs(b2 - a2).max() > 1e-3 * np.abs(a2).max()


def test_layer_head_permutation_invariance():
    """Relabelling the heads in every per-head weight (W_UQ, W_QR, W_UK, W_UV row blocks and
    W_O column blocks) leaves the layer output unchanged: catches a head mixed with another
    head's slice of the output projection."""
    inp = _full_tiny(seed=11)
    d = inp.dims
    perm = [1, 0]

    def rows(w, k):
        return np.concatenate([w[h * k:(h + 1) * k] for h in perm])

    p = dataclasses.replace(
        inp, w_uq=rows(inp.w_uq, d.d_nope), w_qr=rows(inp.w_qr, d.d_rope),
        w_uk=rows(inp.w_uk, d.d_nope), w_uv=rows(inp.w_uv, d.d_v),
        w_o=np.concatenate([inp.w_o[:, h * d.d_v:(h + 1) * d.d_v] for h in perm], axis=1))
    a = O.attention_layer(inp, 0, 4)
    b = O.attention_layer(p, 0, 4)
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-12 * np.abs(a).max())
    assert np.abs(O.attention_layer(dataclasses.replace(p, w_o=inp.w_o), 0, 4) - a).max() > 1e-3
