/*
 * videomla.h -- C ABI of the VideoMLA latent-attention hot path for AMD Instinct MI355X (gfx950).
 *
 * VideoMLA (arXiv 2605.30351) caches, per video token and layer, one head-shared content
 * latent c^KV (Eq. 1) and one head-shared decoupled 3D-RoPE key k^R (Eq. 5) instead of per-head
 * keys and values. A chunk of new tokens attends over a sliding window of cached tokens with
 * FIFO eviction of whole frames (Appendix "Chunk-Causal Sliding-Window Attention"), and at
 * inference the per-head key/value up-projections are absorbed so that attention runs in the
 * latent space (Section "Inference-Time Reparameterization", Eqs. 8-11).
 *
 * Conventions shared by every entry point
 *   - Tensors are device pointers to row-major, contiguous arrays, 16-byte aligned.
 *   - bf16 values are passed as their uint16_t bit patterns.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream). Calls only enqueue work on
 *     it; none synchronizes the host, and none allocates device memory. The caller owns every
 *     buffer: the ring, the workspace, the inputs and the outputs.
 *   - All argument validation happens on the host before any launch. A non-zero return means
 *     nothing was enqueued (except VIDEOMLA_EHIP, which reports a failed launch).
 *   - Thread safety: calls are reentrant; the last error message is thread-local.
 *
 * Token geometry: a latent frame holds grid_h * grid_w tokens in row-major (y, x) order; token n
 * of the chunk whose first frame is frame_end sits at (f, y, x) = (frame_end + n / HW,
 * (n % HW) / grid_w, n % grid_w).
 */
#ifndef VIDEOMLA_H
#define VIDEOMLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define VIDEOMLA_OK 0
#define VIDEOMLA_EINVAL 1       /* NULL pointer, non-positive size, inconsistent dims       */
#define VIDEOMLA_EUNSUPPORTED 2 /* dims the kernels do not tile (see each call)              */
#define VIDEOMLA_EALIGN 3       /* a tensor pointer is not 16-byte aligned                    */
#define VIDEOMLA_EWORKSPACE 4   /* workspace missing or smaller than the size query returned  */
#define VIDEOMLA_EHIP 5         /* a HIP launch failed; the message carries hipGetErrorString */

/*
 * Layer shapes (Section "Method"; Appendix "VideoMLA Block" and "NoPE/RoPE Split and 3D RoPE").
 *   d_model        attention input width d (1536 for Wan2.1-1.3B)
 *   n_heads        n_h (12)
 *   d_nope         per-head content (NoPE) query/key width (paper default 96)
 *   d_rope         width of the head-shared RoPE key and of each head's RoPE query (32)
 *   d_c            latent width of c^KV (192)
 *   d_v            per-head value width, the output width per head (128)
 *   grid_h, grid_w latent tokens per frame = grid_h * grid_w (30 x 52 = 1560)
 *   window_frames  W_f: frames the ring holds, current chunk included (21)
 *   chunk_frames   frames written and attended per call (3)
 *   rope_pairs     complex pairs given to the (t, h, w) axes; 2 * sum = d_rope. Axis t owns the
 *                  first 2 * rope_pairs[0] channels, then h, then w; pair k of an axis is the
 *                  interleaved channel pair (2k, 2k+1) of that axis' slice
 *   rope_band_dim  D_a in theta_{a,k} = rope_base^(-2k / D_a); 0 means 2 * rope_pairs[a]
 *   rope_base      base of the RoPE frequencies (10000)
 *   softmax_scale  multiplier of the scores; 0 means 1 / sqrt(d_nope + d_rope) (Eq. 7)
 *   kv_norm_eps    epsilon of the RMSNorm applied to c^KV when a gain is given
 *   sink_frames    S: leading frames the cache keeps for good (attention sink, App.
 *                  "Chunk-Causal Sliding-Window Attention"); 0 = none. The ring has
 *                  window_frames frame slots: frames 0..S-1 keep slots 0..S-1, later frames
 *                  cycle FIFO through the other window_frames - S slots, which must hold a
 *                  whole chunk (window_frames - S >= chunk_frames).
 *                  RoPE time: with S = 0 keys are rotated at their absolute frame when written
 *                  (a uniform shift of all positions leaves scores unchanged, so this equals a
 *                  window-relative frame). With S > 0 the ring holds UNROTATED keys, and
 *                  videomla_attend rotates the context's keys and the chunk's queries at
 *                  window-local time (App. "Long-Horizon RoPE Re-indexing"): sink frame f at
 *                  t = f, the recent frames in time order at t = S, S+1, ...
 */
typedef struct videomla_dims {
  int32_t d_model, n_heads, d_nope, d_rope, d_c, d_v;
  int32_t grid_h, grid_w;
  int32_t window_frames, chunk_frames;
  int32_t rope_pairs[3];
  int32_t rope_band_dim[3];
  float rope_base;
  float softmax_scale;
  float kv_norm_eps;
  int32_t sink_frames;
} videomla_dims;

/* Host-side window state: absolute index of the first frame of the chunk being generated. */
typedef struct videomla_window {
  int64_t frame_end;
} videomla_window;

/*
 * Options of the attention calls (videomla_attend_ex, videomla_attend_layer,
 * videomla_dense_attend and their workspace-size queries). A NULL options pointer, or a
 * zero-initialized struct, gives the defaults. The library keeps no state between calls: every
 * choice a call depends on is in its arguments, and the adaptive partition keeps its record in
 * the caller's workspace.
 *
 *   n_workgroups   workgroups of the attention kernel; 0 = one per compute unit. The
 *                  (batch, row block, key tile) units are split over them; a row block shared by
 *                  several workgroups leaves one partial result per workgroup, merged exactly by
 *                  their running maxima and sums (the online-softmax merge). Changes the
 *                  workspace size.
 *   partition      VIDEOMLA_PARTITION_EVEN (default): the units are split evenly; outputs are
 *                    bitwise reproducible.
 *                  VIDEOMLA_PARTITION_ADAPTIVE: workgroup k runs on XCD k mod 8, and the XCDs of
 *                    one device can run at different clocks under this load. Each call gives
 *                    each XCD's workgroups a share of the units proportional to the work per
 *                    time that XCD achieved in the previous adaptive call on the same workspace
 *                    (each weight within [0.8, 1.25] of the mean), and records its own times
 *                    there. Split points, and so the rounding of the outputs, can change from
 *                    call to call.
 *                  VIDEOMLA_PARTITION_FROZEN: the weights the last adaptive call on this
 *                    workspace computed (equal weights if there was none), recording nothing:
 *                    outputs are bitwise reproducible from call to call. Calibrate with a few
 *                    adaptive calls, then freeze.
 *                  The state takes 16.4 KB at the end of the workspace. Shapes whose ranges could
 *                  get too short for the workspace's partial-result slots keep the even split.
 *                  Calls that share a workspace must be ordered on one stream.
 *   form           VIDEOMLA_FORM_LATENT (default): the absorbed form (App. "Inference-Time
 *                    Reparameterization", Eqs. 8-11).
 *                  VIDEOMLA_FORM_MATERIALIZED: the training form (Eq. 2, Eq. 7), per-head keys and
 *                    values reconstructed for the window each call (videomla_attend_ex only).
 *                  VIDEOMLA_FORM_AUTO: whichever of the two the library's cost model predicts to
 *                    be faster for (dims, batch, query rows) over a full window; the latent form
 *                    where the materialized one is not built. The choice does not depend on
 *                    frame_end, so the workspace-size query sees the same form.
 *                  Both forms compute the same attention; they differ in rounding only.
 *   query_begin,   the call attends the queries of chunk tokens query_begin ..
 *   query_count      query_begin + query_count - 1 (query_count 0 = to the end of the chunk):
 *                  a block of the chunk's query rows, as one GPU's share of a query-sharded
 *                  chunk, or the few-query regime. q_nope, q_r (q, x) and out (y) then hold
 *                  query_count tokens per batch element, at their chunk positions.
 *   timer          a caller-owned timer (videomla_timer_create), or NULL: each kernel the call
 *                  launches is bracketed by two HIP events recorded on its stream.
 */
#define VIDEOMLA_PARTITION_EVEN 0
#define VIDEOMLA_PARTITION_ADAPTIVE 1
#define VIDEOMLA_PARTITION_FROZEN 2
#define VIDEOMLA_FORM_LATENT 0
#define VIDEOMLA_FORM_MATERIALIZED 1
#define VIDEOMLA_FORM_AUTO 2

typedef struct videomla_timer videomla_timer;

typedef struct videomla_attend_opts {
  int32_t n_workgroups;
  int32_t partition;
  int32_t form;
  int32_t query_begin;
  int32_t query_count;
  videomla_timer* timer;
} videomla_attend_opts;

/*
 * videomla_cache_write -- compress the chunk's tokens and write them into the ring
 * (Eq. 1: c = W_down^KV x; RMSNorm of c when kv_norm_w != NULL; Eq. 5: k^R = W_R^K x rotated by
 * RoPE_3D at the token's absolute (f, y, x); FIFO placement of whole frames).
 *
 *   x          [batch][chunk_frames * HW][d_model]           bf16, chunk tokens in order
 *   w_dkv      [d_c][d_model]                                bf16, W_down^KV
 *   w_kr       [d_rope][d_model]                             bf16, W_R^K
 *   kv_norm_w  [d_c] bf16 RMSNorm gain, or NULL for no normalization
 *   c_kv       [batch][window_frames * HW][d_c]              bf16 ring, written in place
 *   k_r        [batch][window_frames * HW][d_rope]           bf16 ring of ROTATED keys
 *   slots_out  [chunk_frames * HW] int32 slot of each chunk token, or NULL
 * Token (f, y, x) is stored at slot (fs * grid_h + y) * grid_w + x with frame slot
 * fs = f mod window_frames (no sink), or fs = f for f < S and S + (f - S) mod (window_frames - S)
 * otherwise, so the chunk overwrites the oldest non-sink frames; every other slot is left
 * untouched. With a sink, k_r receives the unrotated W_R^K x. Calling it again
 * before videomla_window_advance (the next denoising step) overwrites the same slots.
 * Requires d_model % 64 == 0, d_model <= 2048, d_c % 16 == 0, d_rope % 8 == 0,
 * d_c + d_rope <= 288 (videomla_cache_write_prepared below takes up to 576).
 */
int videomla_cache_write(const videomla_dims* dims, const videomla_window* win, int32_t batch,
                         const uint16_t* x, const uint16_t* w_dkv, const uint16_t* w_kr,
                         const uint16_t* kv_norm_w, uint16_t* c_kv, uint16_t* k_r,
                         int32_t* slots_out, void* stream);

/*
 * The same cache write with the layer's compression weights packed once, at model load, into
 * the order the cache-write kernel consumes them (every token of every call reads the whole
 * [W_down^KV; W_R^K] panel, Eq. 1 and Eq. 5; the packed order lets each GPU load fetch whole
 * cache lines). The values are videomla_cache_write's, up to the order of the fp32 sums.
 *
 * videomla_write_weights_bytes -- size of the packed panel for these dims (0 if the dims are
 *   invalid or not supported by the cache write).
 * videomla_prepare_write_weights -- pack w_dkv [d_c][d_model] and w_kr [d_rope][d_model]
 *   (bf16, as for videomla_cache_write) into w_packed, a caller-owned device buffer of at least
 *   videomla_write_weights_bytes() bytes, 16-byte aligned. Enqueued on `stream`.
 * videomla_cache_write_prepared -- videomla_cache_write with w_packed (as written by
 *   videomla_prepare_write_weights for the same d_model, d_c and d_rope) in place of w_dkv and
 *   w_kr. Same arguments, requirements and errors otherwise, except that d_c + d_rope may be
 *   up to 576 (the d_c = 512 latent of the paper's sweep).
 */
size_t videomla_write_weights_bytes(const videomla_dims* dims);
int videomla_prepare_write_weights(const videomla_dims* dims, const uint16_t* w_dkv,
                                   const uint16_t* w_kr, uint16_t* w_packed, void* stream);
int videomla_cache_write_prepared(const videomla_dims* dims, const videomla_window* win,
                                  int32_t batch, const uint16_t* x, const uint16_t* w_packed,
                                  const uint16_t* kv_norm_w, uint16_t* c_kv, uint16_t* k_r,
                                  int32_t* slots_out, void* stream);

/* Bytes of device workspace videomla_attend needs for this shape and batch (0 if the dims are
 * invalid or not supported); videomla_attend_workspace_bytes_ex for videomla_attend_ex with
 * these options (the form, work partition and query rows change it). */
size_t videomla_attend_workspace_bytes(const videomla_dims* dims, int32_t batch);
size_t videomla_attend_workspace_bytes_ex(const videomla_dims* dims, int32_t batch,
                                          const videomla_attend_opts* opts);

/*
 * videomla_attend -- latent multi-head attention of the chunk's queries over the window.
 * For every batch element b, chunk token n and head h (Section "Inference-Time
 * Reparameterization"):
 *   q_lat   = W_up,h^K^T q_nope[b,n,h]                          (query absorption, Eq. 8)
 *   q_rope  = RoPE_3D(q_r[b,n,h]) at the token's absolute (f, y, x)        (Eq. 6)
 *   s_j     = scale * (q_lat . c_kv[j] + q_rope . k_r[j])                   (Eq. 7)
 *   o_lat   = sum_j softmax(s)_j c_kv[j]   over every valid slot j of the ring
 *   out     = W_up,h^V o_lat                                    (value up-projection, Eq. 2)
 * The valid slots are the first min(window_frames, frame_end + chunk_frames) frame slots:
 * the current chunk (already written by videomla_cache_write), the past frames still held and
 * the sink frames, with no mask (tokens of a chunk see each other; later chunks are not in the
 * ring yet). With a sink, q_r and the ring's keys are rotated at window-local time (see
 * sink_frames) and the workspace also holds the rotated keys.
 *
 *   q_nope  [batch][chunk_frames * HW][n_heads][d_nope]   bf16
 *   q_r     [batch][chunk_frames * HW][n_heads][d_rope]   bf16, unrotated
 *   w_uk    [n_heads * d_nope][d_c]   bf16, W_up^K (head h = rows h*d_nope ..)
 *   w_uv    [n_heads * d_v][d_c]      bf16, W_up^V (head h = rows h*d_v ..)
 *   c_kv, k_r   the rings as written by videomla_cache_write
 *   out     [batch][chunk_frames * HW][n_heads][d_v]      bf16
 *   workspace  device buffer of at least videomla_attend_workspace_bytes() bytes
 * Arithmetic: bf16 operands, fp32 accumulation and softmax, bf16 round-to-nearest-even output.
 * Requires d_nope % 16 == 0 and d_nope <= 128, d_v % 32 == 0 and d_v <= 256,
 * (d_c, d_rope) in {(64, 32), (128, 32), (192, 32), (256, 32), (512, 32), (16, 8)} (the widths
 * of the paper's d_c sweep, Table 5, and a tiny test shape), otherwise VIDEOMLA_EUNSUPPORTED.
 * The work is split evenly over one workgroup per compute unit, so outputs are bitwise
 * reproducible; videomla_attend_ex takes other choices.
 */
int videomla_attend(const videomla_dims* dims, const videomla_window* win, int32_t batch,
                    const uint16_t* q_nope, const uint16_t* q_r, const uint16_t* w_uk,
                    const uint16_t* w_uv, const uint16_t* c_kv, const uint16_t* k_r,
                    uint16_t* out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * videomla_attend_noalloc -- for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): videomla_attend with the
 * same arguments minus the workspace, which is a static device array of the library instead,
 * VIDEOMLA_NOALLOC_SCRATCH_BYTES (64 MiB) on every device it runs on, held until the process
 * ends. Results are videomla_attend's, bit for bit. The call allocates nothing: on its first
 * call on a device it looks up that device's copy of the array. Shapes whose workspace
 * (videomla_attend_workspace_bytes) exceeds the array are rejected with VIDEOMLA_EWORKSPACE
 * before anything is enqueued (the Wan chunk of 4,680 queries needs about 156 MB: use
 * videomla_attend there). Every call on a device shares that device's array: calls that
 * overlap on one device (other streams, other threads) race, so the caller must order them.
 * Nothing in the array needs to start at zero (each call writes what it reads).
 */
#define VIDEOMLA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int videomla_attend_noalloc(const videomla_dims* dims, const videomla_window* win, int32_t batch,
                            const uint16_t* q_nope, const uint16_t* q_r, const uint16_t* w_uk,
                            const uint16_t* w_uv, const uint16_t* c_kv, const uint16_t* k_r,
                            uint16_t* out, void* stream);

/*
 * videomla_attend_ex -- videomla_attend with options (videomla_attend_opts; NULL = the
 * defaults, which make it videomla_attend). With query_begin / query_count, q_nope, q_r and out
 * hold [batch][query_count][n_heads][...] and the queries sit at chunk tokens query_begin ..;
 * the window is the same.
 * With form VIDEOMLA_FORM_MATERIALIZED the attention is computed in the training form (Eq. 2 and
 * Eq. 7; App. "Inference-Time Reparameterization" states that the absorbed form equals it):
 * per-head keys and values are reconstructed for every valid slot of the window,
 *   K_h[j] = [W_up,h^K c_kv[j] ; k_r[j]]  (d_nope + d_rope),   V_h[j] = W_up,h^V c_kv[j]  (d_v),
 * then standard softmax attention runs per head with q = [q_nope ; RoPE_3D(q_r)]. It trades the
 * reconstruction (a GEMM over the window, once per call) for a cheaper score: d_nope + d_rope +
 * d_v multiply-adds per (query, head, key) instead of the latent form's 2 d_c + d_rope; the
 * workspace also holds the reconstructed rows. That form requires d_v == 128, d_nope + d_rope in
 * {128 (the paper's 96 + 32), 160 (128 + 32)}, d_c % 64 == 0 and sink_frames == 0, otherwise
 * VIDEOMLA_EUNSUPPORTED. The workspace must be at least videomla_attend_workspace_bytes_ex()
 * bytes for the same options. EINVAL for options out of range (partition or form unknown,
 * n_workgroups outside [0, 2^20], a query range outside the chunk).
 */
int videomla_attend_ex(const videomla_dims* dims, const videomla_window* win, int32_t batch,
                       const uint16_t* q_nope, const uint16_t* q_r, const uint16_t* w_uk,
                       const uint16_t* w_uv, const uint16_t* c_kv, const uint16_t* k_r,
                       uint16_t* out, void* workspace, size_t workspace_bytes,
                       const videomla_attend_opts* opts, void* stream);

/*
 * The whole attention layer in latent form (App. "Inference-Time Reparameterization",
 * Eqs. 8-11, and App. "VideoMLA Block"): from the chunk's attention input x to the output of
 * the output projection W_O, with the query path absorbed.
 *
 *   c^Q      = RMSNorm(W_down^Q x) with gain gamma_q and eps kv_norm_eps       (Eq. 3)
 *   q_lat_h  = A_h^T c^Q,  A_h = (W_up,h^Q)^T W_up,h^K   [d_q x d_c]           (Eq. 8)
 *   q^rope_h = RoPE_3D(W_R,h^Q c^Q) at the token's position                     (Eq. 6)
 *   o_lat_h  = sum_j softmax_j(scale (q_lat_h . c_j + q^rope_h . k^rope_j)) c_j  (Eqs. 7, 10)
 *   y        = sum_h B_h o_lat_h,  B_h = W_h^O W_up,h^V   [d_model x d_c]       (Eq. 11)
 *
 * A_h and B_h depend only on the weights: videomla_prepare_layer_weights computes them once
 * (fp32 sums, rounded to bf16, the gain gamma_q folded into the query matrices) into an opaque
 * device buffer of videomla_layer_weights_bytes() bytes, which videomla_attend_layer reads.
 */

/* Bytes of the packed layer weights for this shape and query latent width d_q (0 on error). */
size_t videomla_layer_weights_bytes(const videomla_dims* dims, int32_t d_q);

/*
 * videomla_prepare_layer_weights -- pack one layer's weights for videomla_attend_layer.
 *   w_dq     [d_q][d_model]          W_down^Q
 *   gamma_q  [d_q] RMSNorm gain of c^Q, or NULL for ones
 *   w_uq     [n_heads * d_nope][d_q] W_up^Q (head h = rows h*d_nope ..)
 *   w_qr     [n_heads * d_rope][d_q] W_R^Q  (head h = rows h*d_rope ..)
 *   w_uk     [n_heads * d_nope][d_c] W_up^K,  w_uv [n_heads * d_v][d_c] W_up^V
 *   w_o      [d_model][n_heads * d_v] W_O (head h = columns h*d_v ..)
 *   weights  device buffer of at least videomla_layer_weights_bytes() bytes, written
 * Requires d_model % 64 == 0 and 1 <= d_q <= 65536.
 */
int videomla_prepare_layer_weights(const videomla_dims* dims, int32_t d_q, const uint16_t* w_dq,
                                   const uint16_t* gamma_q, const uint16_t* w_uq,
                                   const uint16_t* w_qr, const uint16_t* w_uk,
                                   const uint16_t* w_uv, const uint16_t* w_o, void* weights,
                                   size_t weights_bytes, void* stream);

/* Bytes of device workspace videomla_attend_layer needs for this shape, d_q, batch and options. */
size_t videomla_attend_layer_workspace_bytes(const videomla_dims* dims, int32_t d_q,
                                             int32_t batch, const videomla_attend_opts* opts);

/*
 * videomla_attend_layer -- the layer above for the chunk at win->frame_end, over the same
 * window (and sink context) as videomla_attend.
 *   x        [batch][chunk_frames * HW][d_model]   bf16, the chunk's attention input
 *   weights  as packed by videomla_prepare_layer_weights for the same dims and d_q
 *   c_kv, k_r  the rings as written by videomla_cache_write
 *   y        [batch][chunk_frames * HW][d_model]   bf16, output of the output projection
 * Arithmetic: bf16 operands (c^Q before its normalization, q_cat, o_lat and the packed weights
 * are rounded to bf16), fp32 accumulation, softmax and normalization factors.
 * Requirements of videomla_attend and of videomla_prepare_layer_weights. opts (or NULL) as for
 * videomla_attend_ex, except that the form is always the latent one (form must be LATENT or
 * AUTO); with a query range x and y hold query_count tokens per batch element.
 */
int videomla_attend_layer(const videomla_dims* dims, const videomla_window* win, int32_t batch,
                          int32_t d_q, const uint16_t* x, const void* weights,
                          size_t weights_bytes, const uint16_t* c_kv, const uint16_t* k_r,
                          uint16_t* y, void* workspace, size_t workspace_bytes,
                          const videomla_attend_opts* opts, void* stream);

/*
 * Dense per-head comparator: the cache VideoMLA replaces, built only to measure the latent
 * path against it on the same GPU (per-head keys and values of Eq. 2 without the shared
 * latent; the 3,072-scalar-per-token layout of the Introduction). Head width d = d_v.
 *
 * Full-head 3D RoPE: the d channels of a head are split over (t, h, w) as
 * (d - 4 floor(d/6), 2 floor(d/6), 2 floor(d/6)) channels (44, 42, 42 at d = 128), t first,
 * interleaved pairs as for k^R, each axis with band width D_a equal to its channel count;
 * rope_base is shared with the latent path, dims->rope_pairs and rope_band_dim are ignored.
 */

/* Bytes the dense ring holds per token and layer: 2 * n_heads * d_v * 2 (6,144 B for Wan). */
size_t videomla_dense_cache_bytes_per_token(const videomla_dims* dims);

/*
 * videomla_dense_cache_write -- K_h = W_K,h x rotated by the full-head 3D RoPE at the token's
 * absolute (f, y, x), V_h = W_V,h x, written at the same ring slots as videomla_cache_write.
 *   x          [batch][chunk_frames * HW][d_model]        bf16
 *   w_k, w_v   [n_heads * d_v][d_model]                   bf16 (head h = rows h*d_v ..)
 *   kv         [batch][window_frames * HW][n_heads][2 * d_v]   bf16 ring, written in place:
 *              row (slot, h) holds the rotated K_h, then V_h
 *   slots_out  [chunk_frames * HW] int32, or NULL
 * Arithmetic: bf16 operands, fp32 accumulation and rotation, bf16 round-to-nearest-even.
 * Requires d_model % 64 == 0, d_v % 4 == 0, d_v <= 128, (2 n_heads d_v) % 128 == 0,
 * sink_frames == 0.
 */
int videomla_dense_cache_write(const videomla_dims* dims, const videomla_window* win,
                               int32_t batch, const uint16_t* x, const uint16_t* w_k,
                               const uint16_t* w_v, uint16_t* kv, int32_t* slots_out,
                               void* stream);

/* Bytes of device workspace videomla_dense_attend needs for this shape, batch and options. */
size_t videomla_dense_attend_workspace_bytes(const videomla_dims* dims, int32_t batch,
                                             const videomla_attend_opts* opts);

/*
 * videomla_dense_attend -- standard per-head softmax attention of the chunk's queries over the
 * same window as videomla_attend:
 *   q'   = RoPE_3D,head(q[b,n,h]) at the token's absolute (f, y, x)
 *   out  = sum_j softmax_j(scale * q' . K_h[j]) V_h[j]
 * with scale = softmax_scale, or 1 / sqrt(d_v) when it is 0.
 *   q     [batch][chunk_frames * HW][n_heads][d_v]   bf16, unrotated
 *   kv    the ring as written by videomla_dense_cache_write
 *   out   [batch][chunk_frames * HW][n_heads][d_v]   bf16
 *   workspace  device buffer of at least videomla_dense_attend_workspace_bytes() bytes
 * Arithmetic as videomla_attend. Requires d_v == 128 and sink_frames == 0. opts (or NULL) as
 * for videomla_attend_ex (form ignored); with a query range q and out hold query_count tokens.
 */
int videomla_dense_attend(const videomla_dims* dims, const videomla_window* win, int32_t batch,
                          const uint16_t* q, const uint16_t* kv, uint16_t* out, void* workspace,
                          size_t workspace_bytes, const videomla_attend_opts* opts,
                          void* stream);

/* Slide the window after the last denoising step of a chunk (App. "Chunk-Causal Sliding-Window
 * Attention": each chunk's frames join the window and the oldest frames leave it, first in first
 * out): frame_end += chunk_frames. Host only; the eviction itself is implicit, since the next
 * chunk's videomla_cache_write overwrites the frame slots of the oldest frames. EINVAL for
 * invalid dims or a NULL / negative window. */
int videomla_window_advance(const videomla_dims* dims, videomla_window* win);

/* Bytes the ring holds per token and layer: 2 * (d_c + d_rope), one bf16 latent c^KV and one
 * bf16 decoupled key k^R (Sec. "Compressed KV Cache Construction", Eq. 1 and Eq. 5; the cache
 * traffic per cached token of Eqs. 15-16): 224 scalars = 448 B for Wan against 2 n_h d_h = 3,072
 * for per-head keys and values. 0 for invalid dims. */
size_t videomla_cache_bytes_per_token(const videomla_dims* dims);

/* Number of valid ring slots the chunk at win->frame_end attends over (App. "Chunk-Causal
 * Sliding-Window Attention": the window holds at most window_frames frames, the chunk
 * included): min(window_frames, frame_end + chunk_frames) * HW. Negative on invalid arguments. */
int64_t videomla_valid_tokens(const videomla_dims* dims, const videomla_window* win);

/* Ring slot of the token at absolute position (f, y, x), as videomla_cache_write places it
 * (first-in first-out frame slots, App. "Chunk-Causal Sliding-Window Attention"); negative on
 * invalid arguments. */
int64_t videomla_slot_of(const videomla_dims* dims, int64_t f, int32_t y, int32_t x);

/* Message describing the last non-zero return on this thread ("" if none). */
const char* videomla_last_error(void);

/*
 * Kernel timing with HIP events, for benchmarks. A timer is a caller-owned host object; an
 * attention call whose options name it brackets every kernel it launches (or, after
 * videomla_timer_only, the launches of one kernel) with two events recorded on its stream.
 * videomla_timer_begin / videomla_timer_end bracket whatever the caller enqueues between them on
 * `stream` under one of the names, in the same way (the cache writes, which take no options,
 * are timed like this as "cache_write" and "dense_cache_write"); a begin without its end is
 * dropped by the next begin. After the caller has synchronized the stream, videomla_timer_read
 * accumulates the elapsed time of all completed intervals of one name ("q_absorb",
 * "latent_attend", "out_proj", "rope_window", "bal_prep", "mat_kv", "mat_q_prep", "mat_attend",
 * "mat_merge", "dense_q_prep", "dense_attend", "dense_merge", "q_down", "q_up", "latent_merge",
 * "out_mix", "cache_write", "dense_cache_write") into *count and *total_ms, and forgets them.
 * videomla_timer_only(timer, NULL) times every kernel again; EINVAL for an unknown name or a
 * NULL timer. The events are created without the system-scope fence (GPU-side intervals on one
 * device). A timer may be used by one thread at a time; destroying it releases its events (the
 * caller must have synchronized the streams they were recorded on).
 */
int videomla_timer_create(videomla_timer** timer);
int videomla_timer_destroy(videomla_timer* timer);
int videomla_timer_only(videomla_timer* timer, const char* kernel);
int videomla_timer_begin(videomla_timer* timer, const char* kernel, void* stream);
int videomla_timer_end(videomla_timer* timer, const char* kernel, void* stream);
int videomla_timer_read(videomla_timer* timer, const char* kernel, int64_t* count,
                        double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* VIDEOMLA_H */
