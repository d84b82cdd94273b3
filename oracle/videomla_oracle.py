"""Plain fp64 CPU oracle of the VideoMLA latent-attention hot path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports this module: only the tests, the
package's smoke check and the benchmark's CPU-baseline leg call it. It shares no code with the
HIP kernels or their binding; its only inputs are the seeded bf16 bit patterns that both sides
receive, widened here to fp64.

What it computes, and where the paper defines it (VideoMLA, arXiv 2605.30351):

* compress   c = W_down^KV x (Eq. 1), optional RMSNorm of c (Appendix "VideoMLA Block"),
             k^R = W_R^K x (Eq. 5);
* RoPE_3D    the decoupled (t, h, w) rotary encoding of k^R and q^R (Eqs. 5-6; Appendix
             "NoPE/RoPE Split and 3D RoPE");
* ring slot  where a token's latents live in the sliding-window cache (Appendix "Chunk-Causal
             Sliding-Window Attention": FIFO eviction of whole frames);
* dense      the comparator the latent cache replaces: per-head K = W_K x (rotated by 3D RoPE
             over the whole head) and V = W_V x cached for every token, standard attention;
* layer      the whole attention layer: query latent c^Q = RMSNorm(W_down^Q x), per-head
             queries from it, attention, and the output projection W_O; with the absorbed
             A_h / B_h form of Section "Inference-Time Reparameterization" as a self-check;
* attention  the training-time form: per-head keys/values reconstructed explicitly
             (Eq. 2), score of Eq. 7, softmax over the active window, weighted sum of values.
             Section "Inference-Time Reparameterization" states that the absorbed latent form
             computes exactly this, so the textbook form is the definition the GPU path must
             match. The absorbed form (Eqs. 8-11) is implemented separately as a self-check.

Readings of points the paper leaves open (each is a parameter, never a hidden constant):
RoPE pairs are interleaved channels (2k, 2k+1) of each axis slice, theta_{a,k} = base^(-2k/D_a);
without a sink, keys are rotated at their absolute (f, y, x) when written (a uniform shift of
every position leaves scores unchanged, so this equals the paper's window-relative rotation);
with S sink frames, the cache holds unrotated keys, and the context (sink frames, then the most
recent frames) is rotated at window-local time, the frame's index in the context;
RMSNorm is applied before caching; the softmax scale is 1/sqrt(d_nope + d_rope) (Eq. 7).

Parity pins: every function here is pinned by the `-m "not gpu"` tests against closed forms,
invariants, library routines or printed values of the paper; the fidelity of the RoPE frequency
convention and the RMSNorm epsilon to the trained model is "parity unpinned" (no weights).
"""
from __future__ import annotations

import numpy as np

LOG2E = 1.4426950408889634


# --------------------------------------------------------------------------------------------
# bf16 <-> fp64
# --------------------------------------------------------------------------------------------

def bf16_bits_to_f64(bits) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to fp64, exactly."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def round_to_bf16_bits(v) -> np.ndarray:
    """Round fp64 values to bf16 (nearest, ties to even) in one step; returns uint16 bits.

    bf16 keeps 8 significant bits, so the rounding quantum of v = m * 2^e (0.5 <= |m| < 1) is
    2^(e-8); below the smallest normal (2^-126) the quantum stays at 2^-133.
    """
    v = np.asarray(v, dtype=np.float64)
    _, e = np.frexp(v)
    e = np.maximum(e, -125)
    q = np.ldexp(np.rint(np.ldexp(v, 8 - e)), e - 8)
    return (q.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


# --------------------------------------------------------------------------------------------
# Shapes, positions and the ring slot map
# --------------------------------------------------------------------------------------------

def softmax_scale(dims) -> float:
    """Eq. 7: the joint score is divided by sqrt(d_nope + d_rope)."""
    if dims.softmax_scale and dims.softmax_scale > 0:
        return float(dims.softmax_scale)
    return 1.0 / np.sqrt(dims.d_nope + dims.d_rope)


def cache_scalars_per_token(dims) -> int:
    """Section "Compressed KV Cache Construction": each cached token stores (c^KV, k^R)."""
    return dims.d_c + dims.d_rope


def dense_scalars_per_token(dims) -> int:
    """Dense per-head KV cache of the same backbone: 2 * n_h * d_h, with d_h = d / n_h."""
    return 2 * dims.n_heads * (dims.d_model // dims.n_heads)


def token_position(n, frame_end: int, dims):
    """Token n of the chunk whose first frame is `frame_end`: frames in order, each frame's
    tokens row-major over the (grid_h, grid_w) latent grid. Returns (f, y, x) arrays."""
    n = np.asarray(n, dtype=np.int64)
    f = frame_end + n // dims.hw
    r = n % dims.hw
    return f, r // dims.grid_w, r % dims.grid_w


def frame_slot(f, dims):
    """Frame slot of absolute frame f. Without a sink, frame f lives in slot f mod W_f, so the
    ring holds the most recent W_f frames and the oldest whole frame is evicted first. With S
    sink frames (App. "Chunk-Causal Sliding-Window Attention": one sink frame plus the most
    recent frames, FIFO eviction outside the sink), frames 0..S-1 keep slots 0..S-1 for good and
    later frames cycle through the other W_f - S slots."""
    f = np.asarray(f, dtype=np.int64)
    S, W = dims.sink_frames, dims.window_frames
    if S == 0:
        return f % W
    return np.where(f < S, f, S + (f - S) % (W - S))


def ring_slot(f, y, x, dims):
    """Slot of the token at absolute (f, y, x): its frame slot, then row-major (y, x)."""
    return (frame_slot(f, dims) * dims.grid_h + np.asarray(y)) * dims.grid_w + np.asarray(x)


def window_frame_range(frame_end: int, dims):
    """Frames visible to the chunk starting at `frame_end` when there is no sink: the chunk
    itself plus past frames, at most W_f in total (chunk-causal sliding window).
    Returns [first, last)."""
    assert dims.sink_frames == 0, "a sink context is not a contiguous range: use context_frames"
    last = frame_end + dims.chunk_frames
    return max(0, last - dims.window_frames), last


def context_frames(frame_end: int, dims) -> list:
    """Frames of the active context of the chunk starting at `frame_end`, in time order: the
    sink frames generated so far, then the most recent frames (the chunk included), W_f frames
    at most in total."""
    hi = frame_end + dims.chunk_frames
    S, W = dims.sink_frames, dims.window_frames
    if S == 0:
        return list(range(max(0, hi - W), hi))
    return list(range(min(S, hi))) + list(range(max(S, hi - (W - S)), hi))


def local_time(f, frame_end: int, dims):
    """Window-relative temporal coordinate of context frame f (App. "Long-Horizon RoPE
    Re-indexing"): its index in the context's time order, so the sink frames take 0..S-1 and the
    recent frames follow without a gap. Queries of the chunk take the coordinates of their
    frames. Bounded by W_f - 1 however long the rollout."""
    frames = context_frames(frame_end, dims)
    index = {fr: i for i, fr in enumerate(frames)}
    f = np.asarray(f, dtype=np.int64)
    return np.vectorize(lambda v: index[int(v)], otypes=[np.int64])(f)


# --------------------------------------------------------------------------------------------
# Decoupled 3D RoPE
# --------------------------------------------------------------------------------------------

def rope_axis_layout(dims):
    """Split of the d_rope channels over (t, h, w): axis a owns 2*pairs[a] consecutive channels,
    t first. Returns [(channel_start, n_pairs, band_dim)] for the three axes."""
    pairs = list(dims.rope_pairs)
    assert sum(pairs) * 2 == dims.d_rope, "rope pairs must cover d_rope exactly"
    out, start = [], 0
    for a in range(3):
        band = dims.rope_band_dim[a] if dims.rope_band_dim[a] else 2 * pairs[a]
        out.append((start, pairs[a], band))
        start += 2 * pairs[a]
    return out


def rope3d(v, f, y, x, dims) -> np.ndarray:
    """Rotate each complex pair (2k, 2k+1) of each axis slice of v[..., d_rope] by the angle
    pos_a * base^(-2k / D_a), pos = (f, y, x) broadcast over v's leading dimensions."""
    v = np.asarray(v, dtype=np.float64)
    out = v.copy()
    pos = [np.asarray(f, dtype=np.float64), np.asarray(y, dtype=np.float64),
           np.asarray(x, dtype=np.float64)]
    for a, (start, npairs, band) in enumerate(rope_axis_layout(dims)):
        for k in range(npairs):
            theta = dims.rope_base ** (-2.0 * k / band)
            phi = pos[a] * theta
            while phi.ndim < v.ndim - 1:
                phi = phi[..., None]
            cs, sn = np.cos(phi), np.sin(phi)
            u, w = v[..., start + 2 * k], v[..., start + 2 * k + 1]
            out[..., start + 2 * k] = u * cs - w * sn
            out[..., start + 2 * k + 1] = u * sn + w * cs
    return out


# --------------------------------------------------------------------------------------------
# Cache write: compress, normalize, rotate, place
# --------------------------------------------------------------------------------------------

def compress(x, w_dkv, w_kr, gamma, dims):
    """Eq. 1 and Eq. 5 for a block of tokens x[T, d_model] (fp64): returns (c [T, d_c] after
    the optional RMSNorm with gain gamma, k^R [T, d_rope] unrotated)."""
    c = x @ w_dkv.T
    kr = x @ w_kr.T
    if gamma is not None:
        rms = np.sqrt(np.mean(c * c, axis=-1, keepdims=True) + dims.kv_norm_eps)
        c = gamma * c / rms
    return c, kr


def cache_write(x_chunk_bits, w_dkv_bits, w_kr_bits, gamma_bits, frame_end: int, dims):
    """What `cache_write` must produce for one batch element's chunk.

    x_chunk_bits [chunk_tokens, d_model] bf16 bits of the chunk starting at frame `frame_end`.
    Returns dict: c [T, d_c] fp64; k_cached [T, d_rope] fp64, the positional key as the ring
    holds it: without a sink rotated at the token's absolute (f, y, x) (k_rope, the same array),
    with a sink unrotated (Sec. "Decoupled 3D-RoPE": the cache holds the position-free state,
    rotated when the window is assembled); slots [T] int64.
    """
    x = bf16_bits_to_f64(x_chunk_bits)
    gamma = None if gamma_bits is None else bf16_bits_to_f64(gamma_bits)
    c, kr = compress(x, bf16_bits_to_f64(w_dkv_bits), bf16_bits_to_f64(w_kr_bits), gamma, dims)
    f, y, xx = token_position(np.arange(x.shape[0]), frame_end, dims)
    out = {"c": c, "k_r": kr, "slots": ring_slot(f, y, xx, dims)}
    if dims.sink_frames == 0:
        out["k_rope"] = out["k_cached"] = rope3d(kr, f, y, xx, dims)
    else:
        out["k_cached"] = kr
    return out


def window_latents(x_bits, w_dkv_bits, w_kr_bits, gamma_bits, frame_end: int, dims,
                   rotate_origin: int = 0):
    """Latents of every token visible to the chunk starting at `frame_end`, computed from the
    raw inputs x_bits [n_frames * HW, d_model] (frames from 0), context frames in time order.
    Returns (c, k_rope, (f, y, x)).

    Without a sink, `rotate_origin` is subtracted from every temporal index before rotation
    (0 = absolute positions; the first window frame = the paper's window-relative re-indexing).
    With a sink, keys are rotated at their window-local time (`local_time`)."""
    frames = context_frames(frame_end, dims)
    x = bf16_bits_to_f64(np.concatenate([x_bits[fr * dims.hw:(fr + 1) * dims.hw] for fr in frames]))
    gamma = None if gamma_bits is None else bf16_bits_to_f64(gamma_bits)
    c, kr = compress(x, bf16_bits_to_f64(w_dkv_bits), bf16_bits_to_f64(w_kr_bits), gamma, dims)
    n = np.arange(x.shape[0])
    f = np.asarray(frames, dtype=np.int64)[n // dims.hw]
    y = (n % dims.hw) // dims.grid_w
    xx = n % dims.grid_w
    t = f - rotate_origin if dims.sink_frames == 0 else local_time(f, frame_end, dims)
    return c, rope3d(kr, t, y, xx, dims), (f, y, xx)


# --------------------------------------------------------------------------------------------
# Attention
# --------------------------------------------------------------------------------------------

def _softmax_rows(s):
    m = np.max(s, axis=-1, keepdims=True)
    p = np.exp(s - m)
    return p / np.sum(p, axis=-1, keepdims=True)


def query_positions(rows, frame_end: int, dims):
    """Positions the chunk's query tokens `rows` are rotated at: absolute (f, y, x) without a
    sink, the frames' window-local time with one (the same frame as the context's keys)."""
    f, y, x = token_position(rows, frame_end, dims)
    if dims.sink_frames:
        f = local_time(f, frame_end, dims)
    return f, y, x


def query_rope(q_r, q_pos, dims, rotate_origin: int = 0):
    """Eq. 6: q^rope = RoPE_3D(q^R) at each query token's (f, y, x); q_r [Nq, H, d_rope]."""
    f, y, x = q_pos
    return rope3d(q_r, np.asarray(f) - rotate_origin, y, x, dims)


def attend_unabsorbed(q_nope, q_rope, w_uk, w_uv, c_win, krope_win, dims, row_block=512):
    """Training-time form (Eq. 2 and Eq. 7): per head h reconstruct
    K_h[j] = [W_UK_h c_j ; k^rope_j] and V_h[j] = W_UV_h c_j for every window token j, score
    s_ij = Q_h[i].K_h[j] / sqrt(d_nope + d_rope) with Q_h[i] = [q^nope ; q^rope], softmax over
    all window tokens, o = sum_j p_ij V_h[j].

    q_nope [Nq, H, d_nope], q_rope [Nq, H, d_rope] (already rotated), w_uk [H*d_nope, d_c],
    w_uv [H*d_v, d_c], c_win [S, d_c], krope_win [S, d_rope], all fp64. Returns [Nq, H, d_v].
    Rows are processed in blocks of `row_block` queries only to bound memory.
    """
    nq, H = q_nope.shape[0], dims.n_heads
    scale = softmax_scale(dims)
    out = np.empty((nq, H, dims.d_v))
    for h in range(H):
        w_uk_h = w_uk[h * dims.d_nope:(h + 1) * dims.d_nope]      # [d_nope, d_c]
        w_uv_h = w_uv[h * dims.d_v:(h + 1) * dims.d_v]            # [d_v, d_c]
        k_h = np.concatenate([c_win @ w_uk_h.T, krope_win], axis=1)
        v_h = c_win @ w_uv_h.T
        for r0 in range(0, nq, row_block):
            q_h = np.concatenate([q_nope[r0:r0 + row_block, h], q_rope[r0:r0 + row_block, h]],
                                 axis=1)
            p = _softmax_rows(scale * (q_h @ k_h.T))
            out[r0:r0 + row_block, h] = p @ v_h
    return out


def attend_absorbed(q_nope, q_rope, w_uk, w_uv, c_win, krope_win, dims):
    """Inference-time form (Eqs. 8-11, in the per-head-query form): q_lat = W_UK_h^T q^nope,
    score (q_lat.c_j + q^rope.k^rope_j) * scale, o_lat = sum_j p_ij c_j, o = W_UV_h o_lat.
    Self-check only: it must equal `attend_unabsorbed` up to rounding."""
    nq, H = q_nope.shape[0], dims.n_heads
    scale = softmax_scale(dims)
    out = np.empty((nq, H, dims.d_v))
    for h in range(H):
        w_uk_h = w_uk[h * dims.d_nope:(h + 1) * dims.d_nope]
        w_uv_h = w_uv[h * dims.d_v:(h + 1) * dims.d_v]
        q_lat = q_nope[:, h] @ w_uk_h                              # [Nq, d_c]
        p = _softmax_rows(scale * (q_lat @ c_win.T + q_rope[:, h] @ krope_win.T))
        out[:, h] = (p @ c_win) @ w_uv_h.T
    return out


def chunk_attention(inp, b: int, frame_end: int, rows=None, absorbed: bool = False,
                    rotate_origin: int | None = None):
    """End-to-end reference for one batch element: the chunk starting at `frame_end` attends
    over its window, every latent computed from the raw inputs in fp64.

    `inp` is a workloads.LayerInputs; `rows` optionally selects query tokens of the chunk.
    `rotate_origin` None = absolute positions; otherwise positions are shifted by that amount
    for both queries and keys. Returns [len(rows), H, d_v] fp64.
    """
    dims = inp.dims
    origin = 0 if rotate_origin is None else rotate_origin
    c_win, kro_win, _ = window_latents(inp.x[b], inp.w_dkv, inp.w_kr, inp.gamma, frame_end, dims,
                                       rotate_origin=origin)
    rows = np.arange(dims.chunk_tokens) if rows is None else np.asarray(rows)
    q_nope = bf16_bits_to_f64(inp.q_nope[b][rows])
    q_pos = query_positions(rows, frame_end, dims)
    if dims.sink_frames:
        origin = 0
    q_rope = query_rope(bf16_bits_to_f64(inp.q_r[b][rows]), q_pos, dims, rotate_origin=origin)
    w_uk, w_uv = bf16_bits_to_f64(inp.w_uk), bf16_bits_to_f64(inp.w_uv)
    fn = attend_absorbed if absorbed else attend_unabsorbed
    return fn(q_nope, q_rope, w_uk, w_uv, c_win, kro_win, dims)


# --------------------------------------------------------------------------------------------
# Whole attention layer: query path and output projection
# --------------------------------------------------------------------------------------------

def rms_norm(v, gain, eps):
    """RMSNorm over the last axis: gain * v / sqrt(mean(v^2) + eps) (App. "VideoMLA Block":
    c^KV and c^Q are normalized before their up-projections)."""
    return gain * v / np.sqrt(np.mean(v * v, axis=-1, keepdims=True) + eps)


def query_latent(x, w_dq, gamma_q, dims):
    """c^Q = RMSNorm(W_down^Q x) for tokens x[T, d_model] (Eq. 3), fp64."""
    return rms_norm(x @ w_dq.T, gamma_q, dims.kv_norm_eps)


def attention_layer(inp, b: int, frame_end: int, rows=None):
    """The whole attention layer for the chunk starting at `frame_end`, training-time form:
    c^Q (Eq. 3); per head q^nope = W_up,h^Q c^Q (Eq. 4) and q^R = W_R,h^Q c^Q rotated (Eq. 6);
    keys and values reconstructed from the window latents (Eq. 2); scores of Eq. 7, softmax over
    the window; the head outputs concatenated and mixed by W_O. `inp` is a
    workloads.FullLayerInputs. Returns y [len(rows), d_model] fp64."""
    d = inp.dims
    rows = np.arange(d.chunk_tokens) if rows is None else np.asarray(rows)
    x = bf16_bits_to_f64(inp.x[b][frame_end * d.hw:(frame_end + d.chunk_frames) * d.hw][rows])
    cq = query_latent(x, bf16_bits_to_f64(inp.w_dq), bf16_bits_to_f64(inp.gamma_q), d)
    n, H = len(rows), d.n_heads
    q_nope = (cq @ bf16_bits_to_f64(inp.w_uq).T).reshape(n, H, d.d_nope)
    q_r = (cq @ bf16_bits_to_f64(inp.w_qr).T).reshape(n, H, d.d_rope)
    q_rope = query_rope(q_r, query_positions(rows, frame_end, d), d)
    c_win, kro_win, _ = window_latents(inp.x[b], inp.w_dkv, inp.w_kr, inp.gamma, frame_end, d)
    o = attend_unabsorbed(q_nope, q_rope, bf16_bits_to_f64(inp.w_uk), bf16_bits_to_f64(inp.w_uv),
                          c_win, kro_win, d)
    return o.reshape(n, H * d.d_v) @ bf16_bits_to_f64(inp.w_o).T


def absorbed_layer_weights(inp):
    """App. "Inference-Time Reparameterization": A_h = (W_up,h^Q)^T W_up,h^K [d_q, d_c] and
    B_h = W_h^O W_up,h^V [d_model, d_c] for every head, fp64. Returns (A [H, d_q, d_c],
    B [H, d_model, d_c])."""
    d = inp.dims
    w_uq, w_uk = bf16_bits_to_f64(inp.w_uq), bf16_bits_to_f64(inp.w_uk)
    w_uv, w_o = bf16_bits_to_f64(inp.w_uv), bf16_bits_to_f64(inp.w_o)
    A = np.stack([w_uq[h * d.d_nope:(h + 1) * d.d_nope].T @ w_uk[h * d.d_nope:(h + 1) * d.d_nope]
                  for h in range(d.n_heads)])
    B = np.stack([w_o[:, h * d.d_v:(h + 1) * d.d_v] @ w_uv[h * d.d_v:(h + 1) * d.d_v]
                  for h in range(d.n_heads)])
    return A, B


def attention_layer_absorbed(inp, b: int, frame_end: int, rows=None):
    """The same layer in latent form (Eqs. 8-11): content score (c^Q)^T A_h c_j, positional
    score q^rope . k^rope_j, o_lat = sum_j p_j c_j, y = sum_h B_h o_lat_h. Self-check only: it
    must equal `attention_layer` up to rounding."""
    d = inp.dims
    rows = np.arange(d.chunk_tokens) if rows is None else np.asarray(rows)
    x = bf16_bits_to_f64(inp.x[b][frame_end * d.hw:(frame_end + d.chunk_frames) * d.hw][rows])
    cq = query_latent(x, bf16_bits_to_f64(inp.w_dq), bf16_bits_to_f64(inp.gamma_q), d)
    n, H = len(rows), d.n_heads
    q_r = (cq @ bf16_bits_to_f64(inp.w_qr).T).reshape(n, H, d.d_rope)
    q_rope = query_rope(q_r, query_positions(rows, frame_end, d), d)
    c_win, kro_win, _ = window_latents(inp.x[b], inp.w_dkv, inp.w_kr, inp.gamma, frame_end, d)
    A, B = absorbed_layer_weights(inp)
    scale = softmax_scale(d)
    y = np.zeros((n, d.d_model))
    for h in range(H):
        p = _softmax_rows(scale * ((cq @ A[h]) @ c_win.T + q_rope[:, h] @ kro_win.T))
        y += (p @ c_win) @ B[h].T
    return y


# --------------------------------------------------------------------------------------------
# Dense per-head comparator: the cache VideoMLA replaces (Sec. "Introduction" and Table 3's
# dense-KV baseline; Eq. 2 without the shared latent)
# --------------------------------------------------------------------------------------------

def dense_head_rope_dims(dims):
    """RoPE geometry of a full dense head of width d = d_v: the Wan split of a head's channels
    over (t, h, w), (d - 4*floor(d/6), 2*floor(d/6), 2*floor(d/6)) channels, with each axis'
    band width equal to its channel count. At d = 128 this is (44, 42, 42) channels, the groups
    the paper takes its RoPE key bands from (App. "NoPE/RoPE Split and 3D RoPE")."""
    d = dims.d_v
    k = d // 6
    ch = (d - 4 * k, 2 * k, 2 * k)
    return dims.replace(d_rope=d, rope_pairs=tuple(c // 2 for c in ch), rope_band_dim=ch)


def dense_kv(x, w_k, w_v, pos, dims):
    """Per-head keys and values of tokens x[T, d_model] (fp64): K_h = W_K,h x rotated by 3D
    RoPE over the whole head at pos = (f, y, x), V_h = W_V,h x. w_k, w_v [H*d_v, d_model].
    Returns (K [T, H, d_v], V [T, H, d_v])."""
    T, H, d = x.shape[0], dims.n_heads, dims.d_v
    k = (x @ w_k.T).reshape(T, H, d)
    v = (x @ w_v.T).reshape(T, H, d)
    f, y, xx = pos
    hd = dense_head_rope_dims(dims)
    k = rope3d(k, np.asarray(f)[:, None], np.asarray(y)[:, None], np.asarray(xx)[:, None], hd)
    return k, v


def dense_cache_write(x_chunk_bits, w_k_bits, w_v_bits, frame_end: int, dims):
    """What the dense comparator's cache write must produce for one batch element's chunk:
    rotated keys, values and the slots (the same FIFO ring placement as the latent cache)."""
    x = bf16_bits_to_f64(x_chunk_bits)
    pos = token_position(np.arange(x.shape[0]), frame_end, dims)
    k, v = dense_kv(x, bf16_bits_to_f64(w_k_bits), bf16_bits_to_f64(w_v_bits), pos, dims)
    return {"k": k, "v": v, "slots": ring_slot(*pos, dims)}


def dense_attend(q, k_win, v_win, q_pos, dims, row_block=512):
    """Standard per-head attention of queries q [Nq, H, d_v] (unrotated) over window keys
    k_win [S, H, d_v] (rotated) and values v_win [S, H, d_v]: q rotated by the full-head RoPE
    at q_pos, scores scaled by 1/sqrt(d_v) (or dims.softmax_scale when given), softmax over the
    window. Returns [Nq, H, d_v] fp64."""
    hd = dense_head_rope_dims(dims)
    f, y, x = q_pos
    qr = rope3d(q, np.asarray(f)[:, None], np.asarray(y)[:, None], np.asarray(x)[:, None], hd)
    scale = dims.softmax_scale if dims.softmax_scale else 1.0 / np.sqrt(dims.d_v)
    nq, H = q.shape[0], dims.n_heads
    out = np.empty((nq, H, dims.d_v))
    for h in range(H):
        for r0 in range(0, nq, row_block):
            p = _softmax_rows(scale * (qr[r0:r0 + row_block, h] @ k_win[:, h].T))
            out[r0:r0 + row_block, h] = p @ v_win[:, h]
    return out


def dense_chunk_attention(inp, b: int, frame_end: int, rows=None):
    """End-to-end dense reference for one batch element (inp: workloads.DenseInputs)."""
    dims = inp.dims
    lo, hi = window_frame_range(frame_end, dims)
    x = bf16_bits_to_f64(inp.x[b][lo * dims.hw: hi * dims.hw])
    n = np.arange(x.shape[0])
    pos = (lo + n // dims.hw, (n % dims.hw) // dims.grid_w, n % dims.grid_w)
    k, v = dense_kv(x, bf16_bits_to_f64(inp.w_k), bf16_bits_to_f64(inp.w_v), pos, dims)
    rows = np.arange(dims.chunk_tokens) if rows is None else np.asarray(rows)
    q = bf16_bits_to_f64(inp.q[b][rows])
    return dense_attend(q, k, v, token_position(rows, frame_end, dims), dims)


def ring_after_writes(n_frames_written: int, dims):
    """Absolute frame held by each frame slot after frames 0 .. n_frames_written-1 were written
    in order (-1 = never written). Follows the closed-form slot map."""
    held = np.full(dims.window_frames, -1, dtype=np.int64)
    for f in range(n_frames_written):
        held[int(frame_slot(f, dims))] = f
    return held
