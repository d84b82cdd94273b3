"""Workload shapes and seeded synthetic inputs for the VideoMLA latent-attention path.

This module is shared by the tests, the benchmark and the CPU oracle's callers. It holds only
shapes and random-number generation: none of the method's arithmetic lives here, so the oracle
and the HIP path stay independent of each other.

Token geometry follows the paper's Wan2.1-T2V-1.3B setting (Appendix "Backbone and
Tokenization"): 832x480 video, 30x52 = 1560 latent tokens per frame, chunks of 3 latent frames,
a 21-frame window. Weights follow N(0, std = 1/sqrt(fan_in)); activations N(0, 1); all values are
drawn in float32 from numpy's PCG64 and rounded to bf16 with round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Dims:
    """Layer shapes; mirrors the `videomla_dims` struct of the C ABI field by field."""

    d_model: int
    n_heads: int
    d_nope: int
    d_rope: int
    d_c: int
    d_v: int
    grid_h: int
    grid_w: int
    window_frames: int
    chunk_frames: int
    rope_pairs: tuple = (0, 0, 0)          # complex pairs per (t, h, w) axis; sum = d_rope / 2
    rope_band_dim: tuple = (0, 0, 0)       # D_a in theta = base^(-2k/D_a); 0 means 2 * pairs
    rope_base: float = 10000.0
    softmax_scale: float = 0.0             # 0 means 1/sqrt(d_nope + d_rope)
    kv_norm_eps: float = 1e-6
    sink_frames: int = 0                   # leading frames kept for good (attention sink)

    @property
    def hw(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def chunk_tokens(self) -> int:
        return self.chunk_frames * self.hw

    @property
    def window_tokens(self) -> int:
        return self.window_frames * self.hw

    def replace(self, **kw) -> "Dims":
        return dataclasses.replace(self, **kw)


# Tiny case: 2 heads, d_c = 16, d_rope = 8, 4x4 grid, 3-frame window, 1-frame chunks.
TINY = Dims(d_model=64, n_heads=2, d_nope=32, d_rope=8, d_c=16, d_v=32, grid_h=4, grid_w=4,
            window_frames=3, chunk_frames=1, rope_pairs=(2, 1, 1))

# Wan2.1-1.3B layer as measured: d_nope = 128, RoPE channels t:16 h:8 w:8 (pairs 8, 4, 4).
WAN = Dims(d_model=1536, n_heads=12, d_nope=128, d_rope=32, d_c=192, d_v=128, grid_h=30,
           grid_w=52, window_frames=21, chunk_frames=3, rope_pairs=(8, 4, 4))

# The paper's own default split: d_nope = 96, (6, 5, 5) pairs taken from the highest-frequency
# bands of Wan's full-head axis groups (44, 42, 42 channels).
WAN_PAPER = WAN.replace(d_nope=96, rope_pairs=(6, 5, 5), rope_band_dim=(44, 42, 42))

# The paper's long-rollout context: one sink frame and the six most recent frames (7 frame
# slots, 10,920 cached tokens); keys are cached unrotated and rotated in window-local time.
WAN_SINK = WAN.replace(window_frames=7, sink_frames=1)

# Tiny sink case: one sink frame and three local frames, 1-frame chunks.
TINY_SINK = TINY.replace(window_frames=4, sink_frames=1)

# The latent widths of the paper's d_c sweep (Table 5), Wan geometry otherwise.
DC_SWEEP = (64, 128, 192, 256, 512)
WAN_DC = {dc: WAN.replace(d_c=dc) for dc in DC_SWEEP}

# Few-query regime: 1-frame chunks (1,560 queries per call) over the 21-frame window.
WAN_1F = WAN.replace(chunk_frames=1)

# A small shape with Wan's head and RoPE widths: 2 heads, a 6x10 grid, a 5-frame window (300
# keys: a ragged last key tile) and 2-frame chunks (120 queries); d_c is set per case.
SMALL = Dims(d_model=256, n_heads=2, d_nope=128, d_rope=32, d_c=192, d_v=128, grid_h=6,
             grid_w=10, window_frames=5, chunk_frames=2, rope_pairs=(8, 4, 4))

# SMALL with the paper's own head split (d_nope 96 + d_rope 32 = d_v = 128).
SMALL_PAPER = SMALL.replace(d_nope=96, rope_pairs=(6, 5, 5), rope_band_dim=(44, 42, 42))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    v = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        v *= np.float32(std)
    return f32_to_bf16_bits(v)


@dataclass
class LayerInputs:
    """One layer's seeded inputs, all bf16 bit patterns (uint16), row-major.

    x       [batch, n_frames * HW, d_model]   frames 0 .. n_frames-1, token order (f, y, x)
    w_dkv   [d_c, d_model]                    KV down-projection
    w_kr    [d_rope, d_model]                 decoupled RoPE key projection
    w_uk    [n_heads * d_nope, d_c]           key up-projection, head h = rows h*d_nope ..
    w_uv    [n_heads * d_v, d_c]              value up-projection, head h = rows h*d_v ..
    gamma   [d_c] or None                     RMSNorm gain on the latent (None = no norm)
    q_nope  [batch, chunk_tokens, n_heads, d_nope]   queries of the chunk being denoised
    q_r     [batch, chunk_tokens, n_heads, d_rope]   unrotated positional queries
    """

    dims: Dims
    batch: int
    n_frames: int
    x: np.ndarray
    w_dkv: np.ndarray
    w_kr: np.ndarray
    w_uk: np.ndarray
    w_uv: np.ndarray
    gamma: np.ndarray | None
    q_nope: np.ndarray
    q_r: np.ndarray
    meta: dict = field(default_factory=dict)


def make_layer_inputs(dims: Dims, seed: int, n_frames: int, batch: int = 1, norm: bool = True,
                      q_gain: float = 1.0, random_gain: bool = False) -> LayerInputs:
    """Draw one layer's inputs in a fixed order: x frames, W_DKV, W_KR, W_UK, W_UV, q_nope, q_R.

    `q_gain` multiplies the float32 query draws before rounding (4.0 gives the peaked-softmax
    variant whose scaled scores have std of about 4). With `norm`, the RMSNorm gain is all ones,
    or with `random_gain` drawn uniform in [0.5, 1.5) from a stream of its own (seed, 7), so that
    the other draws are the same either way.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    d = dims
    x = _normal_bf16(rng, (batch, n_frames * d.hw, d.d_model))
    w_dkv = _normal_bf16(rng, (d.d_c, d.d_model), 1.0 / np.sqrt(d.d_model))
    w_kr = _normal_bf16(rng, (d.d_rope, d.d_model), 1.0 / np.sqrt(d.d_model))
    w_uk = _normal_bf16(rng, (d.n_heads * d.d_nope, d.d_c), 1.0 / np.sqrt(d.d_c))
    w_uv = _normal_bf16(rng, (d.n_heads * d.d_v, d.d_c), 1.0 / np.sqrt(d.d_c))
    gamma = f32_to_bf16_bits(np.ones(d.d_c, np.float32)) if norm else None
    if norm and random_gain:
        g_rng = np.random.Generator(np.random.PCG64([seed, 7]))
        gamma = f32_to_bf16_bits(g_rng.uniform(0.5, 1.5, size=d.d_c).astype(np.float32))
    qn = rng.standard_normal(size=(batch, d.chunk_tokens, d.n_heads, d.d_nope), dtype=np.float32)
    qr = rng.standard_normal(size=(batch, d.chunk_tokens, d.n_heads, d.d_rope), dtype=np.float32)
    if q_gain != 1.0:
        qn *= np.float32(q_gain)
        qr *= np.float32(q_gain)
    return LayerInputs(d, batch, n_frames, x, w_dkv, w_kr, w_uk, w_uv, gamma,
                       f32_to_bf16_bits(qn), f32_to_bf16_bits(qr))


@dataclass
class FullLayerInputs:
    """Seeded inputs of a whole attention layer: the cache path of LayerInputs plus the query
    path and the output projection (App. "VideoMLA Block"), bf16 bit patterns.

    x, w_dkv, w_kr, w_uk, w_uv, gamma   as in LayerInputs (gamma: RMSNorm gain of c^KV)
    w_dq     [d_q, d_model]               query down-projection W_down^Q
    gamma_q  [d_q]                        RMSNorm gain of c^Q
    w_uq     [n_heads * d_nope, d_q]      query up-projection W_up^Q, head h = rows h*d_nope ..
    w_qr     [n_heads * d_rope, d_q]      RoPE query projection W_R^Q, head h = rows h*d_rope ..
    w_o      [d_model, n_heads * d_v]     output projection W_O, head h = columns h*d_v ..
    """

    dims: Dims
    batch: int
    n_frames: int
    d_q: int
    x: np.ndarray
    w_dkv: np.ndarray
    w_kr: np.ndarray
    w_uk: np.ndarray
    w_uv: np.ndarray
    gamma: np.ndarray | None
    w_dq: np.ndarray
    gamma_q: np.ndarray
    w_uq: np.ndarray
    w_qr: np.ndarray
    w_o: np.ndarray


def make_full_layer_inputs(dims: Dims, seed: int, n_frames: int, d_q: int,
                           batch: int = 1) -> FullLayerInputs:
    """Draw a whole layer's inputs in a fixed order: x frames, W_DKV, W_KR, W_UK, W_UV (as
    make_layer_inputs), then W_DQ, the c^Q gain (uniform in [0.5, 1.5], so that folding it into
    the query weights is exercised), W_UQ, W_QR, W_O."""
    rng = np.random.Generator(np.random.PCG64(seed))
    d = dims
    x = _normal_bf16(rng, (batch, n_frames * d.hw, d.d_model))
    w_dkv = _normal_bf16(rng, (d.d_c, d.d_model), 1.0 / np.sqrt(d.d_model))
    w_kr = _normal_bf16(rng, (d.d_rope, d.d_model), 1.0 / np.sqrt(d.d_model))
    w_uk = _normal_bf16(rng, (d.n_heads * d.d_nope, d.d_c), 1.0 / np.sqrt(d.d_c))
    w_uv = _normal_bf16(rng, (d.n_heads * d.d_v, d.d_c), 1.0 / np.sqrt(d.d_c))
    gamma = f32_to_bf16_bits(np.ones(d.d_c, np.float32))
    w_dq = _normal_bf16(rng, (d_q, d.d_model), 1.0 / np.sqrt(d.d_model))
    gamma_q = f32_to_bf16_bits(rng.uniform(0.5, 1.5, size=d_q).astype(np.float32))
    w_uq = _normal_bf16(rng, (d.n_heads * d.d_nope, d_q), 1.0 / np.sqrt(d_q))
    w_qr = _normal_bf16(rng, (d.n_heads * d.d_rope, d_q), 1.0 / np.sqrt(d_q))
    w_o = _normal_bf16(rng, (d.d_model, d.n_heads * d.d_v), 1.0 / np.sqrt(d.n_heads * d.d_v))
    return FullLayerInputs(d, batch, n_frames, d_q, x, w_dkv, w_kr, w_uk, w_uv, gamma, w_dq,
                           gamma_q, w_uq, w_qr, w_o)


@dataclass
class DenseInputs:
    """Seeded inputs of the dense per-head comparator (bf16 bit patterns).

    x      [batch, n_frames * HW, d_model]   token activations
    w_k    [n_heads * d_v, d_model]          per-head key projection
    w_v    [n_heads * d_v, d_model]          per-head value projection
    q      [batch, chunk_tokens, n_heads, d_v]   unrotated queries of the chunk
    """

    dims: Dims
    batch: int
    n_frames: int
    x: np.ndarray
    w_k: np.ndarray
    w_v: np.ndarray
    q: np.ndarray


def make_dense_inputs(dims: Dims, seed: int, n_frames: int, batch: int = 1) -> DenseInputs:
    """Draw the comparator's inputs in a fixed order: x frames, W_K, W_V, q."""
    rng = np.random.Generator(np.random.PCG64(seed))
    d = dims
    x = _normal_bf16(rng, (batch, n_frames * d.hw, d.d_model))
    w_k = _normal_bf16(rng, (d.n_heads * d.d_v, d.d_model), 1.0 / np.sqrt(d.d_model))
    w_v = _normal_bf16(rng, (d.n_heads * d.d_v, d.d_model), 1.0 / np.sqrt(d.d_model))
    q = _normal_bf16(rng, (batch, d.chunk_tokens, d.n_heads, d.d_v))
    return DenseInputs(d, batch, n_frames, x, w_k, w_v, q)


def chunk_frame_ends(dims: Dims, n_frames: int) -> list[int]:
    """First frame of each chunk when frames 0 .. n_frames-1 are written chunk by chunk."""
    assert n_frames % dims.chunk_frames == 0
    return list(range(0, n_frames, dims.chunk_frames))
