"""A CPU model of the attention path's bf16 storage points, for tests.

The HIP path keeps these values in bf16 (round to nearest even): the ring (c^KV and the rotated
k^R), the absorbed query rows (q_lat and q^rope, both scaled by softmax scale x log2 e), the
probabilities the value product multiplies (and sums, for the softmax denominator), the merged
latent o_lat, and the output; every sum is exact here. The model computes the latent attention
(the absorbed form of App. "Inference-Time Reparameterization", Eqs. 8-11) in float64 from the
oracle's own functions with exactly those values rounded and nothing else, so its error against
the fp64 oracle is the error that bf16 storage alone admits on a given input.

It is not the kernel: the kernel's running maximum is raised lazily, so its probabilities are
2^(s - m) for an m up to 8 below the row maximum and round differently, and its fp32 sums are
not exact. It serves to bound what any implementation with this storage precision can reach on
shapes where that bound exceeds the fixed tolerance (one query row per call).
"""
import numpy as np

from oracle import videomla_oracle as O


def bf16(v):
    """Round float64 values to bf16 (nearest even) and back."""
    return O.bf16_bits_to_f64(O.round_to_bf16_bits(np.asarray(v, dtype=np.float64)))


def chunk_attention_bf16_storage(inp, b: int, frame_end: int):
    """The attention of the chunk at `frame_end` (batch element b, no sink) with the path's
    storage points rounded to bf16; [chunk_tokens, H, d_v] float64."""
    d = inp.dims
    assert d.sink_frames == 0
    c, kr, _ = O.window_latents(inp.x[b], inp.w_dkv, inp.w_kr, inp.gamma, frame_end, d)
    c, kr = bf16(c), bf16(kr)
    rows = np.arange(d.chunk_tokens)
    qn = O.bf16_bits_to_f64(inp.q_nope[b][rows])
    qr = O.query_rope(O.bf16_bits_to_f64(inp.q_r[b][rows]), O.query_positions(rows, frame_end, d),
                      d)
    w_uk, w_uv = O.bf16_bits_to_f64(inp.w_uk), O.bf16_bits_to_f64(inp.w_uv)
    sc = O.softmax_scale(d) * np.log2(np.e)
    out = np.empty((d.chunk_tokens, d.n_heads, d.d_v))
    for h in range(d.n_heads):
        q_lat = bf16(qn[:, h] @ w_uk[h * d.d_nope:(h + 1) * d.d_nope] * sc)
        q_rope = bf16(qr[:, h] * sc)
        s = q_lat @ c.T + q_rope @ kr.T                     # log2 units
        p = bf16(np.exp2(s - s.max(axis=1, keepdims=True)))
        o_lat = bf16((p @ c) / p.sum(axis=1, keepdims=True))
        out[:, h] = bf16(o_lat @ w_uv[h * d.d_v:(h + 1) * d.d_v].T)
    return out


def storage_bars(inp, b: int, frame_end: int, want, factor: float = 1.5):
    """(max-abs, mean-abs, relative L2) bars for one call: the fixed tolerance (2e-2, 2e-3,
    1e-2), or `factor` times the model's own error against the oracle output `want` where that
    is larger."""
    got = chunk_attention_bf16_storage(inp, b, frame_end)
    err = np.abs(got - want)
    rel = np.linalg.norm(got - want) / np.linalg.norm(want)
    return max(2e-2, factor * err.max()), max(2e-3, factor * err.mean()), max(1e-2, factor * rel)
