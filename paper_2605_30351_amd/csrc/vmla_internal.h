// Launch arguments shared by the C-ABI layer (videomla_api.cpp) and the kernel files.
// Host-visible plain structs only; no device code here.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vmla {

constexpr int kMaxRopePairs = 64;  // a whole dense head of 128 channels
constexpr int kMaxWriteDModel = 2048;  // cache write: 32 resident x rows of d_model fill 128 KB of LDS
constexpr int kMaxWriteOutPlain = 288;   // d_c + d_rope of the plain-weight cache write
constexpr int kMaxWriteOutPacked = 576;  // d_c + d_rope of the packed-weight cache write
// 16-row output blocks per wave of the packed-weight cache write: 2 (32 outputs) up to 288
// outputs, else 4 (64 outputs), so that at most 9 waves cover d_c + d_rope
__host__ __device__ inline int write_blocks_per_wave(int outputs) { return outputs <= kMaxWriteOutPlain ? 2 : 4; }

// Per RoPE pair p (interleaved channels 2p, 2p+1 of the d_rope vector): the axis whose
// coordinate drives it (0 = t, 1 = h, 2 = w) and theta = base^(-2k / D_axis), in double.
struct RopeTable {
  int32_t n_pairs;
  int32_t axis[kMaxRopePairs];
  double theta[kMaxRopePairs];
};

struct Geometry {
  int32_t grid_h, grid_w, window_frames;
  int32_t chunk_tokens;   // chunk_frames * HW
  // Queries of an attention call: chunk tokens q_begin .. q_begin + q_count - 1 (the whole
  // chunk unless the call asks for a block of its query rows); q_count tokens per batch element
  // in the query, output and workspace tensors.
  int32_t q_begin, q_count;
  int64_t frame_end;      // absolute first frame of the chunk
  int64_t ring_tokens;    // window_frames * HW (ring rows per batch element)
  // Attention sink: frames 0 .. sink_frames-1 keep frame slots 0 .. sink_frames-1, later frames
  // cycle through the other window_frames - sink_frames slots. With a sink, positional keys are
  // cached unrotated and the context is rotated at window-local time: frame f < sink_frames at
  // f, a recent frame f at sink_frames + (f - local_lo).
  int32_t sink_frames;
  int64_t local_lo;       // first recent frame of the chunk's context (sink_frames > 0 only)
};

#ifdef VMLA_PHASE_STAMPS
// Phase stamps, in the diagnostic build only (the same sources compiled with
// VMLA_PHASE_STAMPS into libvideomla_stamps.so). Lane 0 of every wave of the stamped kernels
// writes the 100 MHz real-time counter at named points of the kernel into a caller-owned
// device buffer of uint64 [kernel][workgroup][wave][point]; the launch arguments carry the
// buffer that videomla_stamps_attach last set. The product build has neither the field nor
// the stores.
constexpr int kStampKernels = 5, kStampWorkgroups = 2048, kStampWaves = 8, kStampPoints = 16;
constexpr int64_t kStampBufferBytes =
    (int64_t)kStampKernels * kStampWorkgroups * kStampWaves * kStampPoints * 8;
enum StampKernel {
  kStampWritePacked = 0,  // cache_write_packed_kernel
  kStampWriteWide = 1,    // cache_write_wide_kernel
  kStampQAbsorb = 2,      // q_absorb_kernel
  kStampAttend = 3,       // latent_attend_kernel (latent form)
  kStampOutProj = 4,      // out_proj_kernel
};
uint64_t* stamp_buffer();  // the attached buffer, or nullptr (videomla_api.cpp)
#endif

struct WriteArgs {
#ifdef VMLA_PHASE_STAMPS
  uint64_t* stamps = stamp_buffer();
#endif
  const uint16_t* x;      // [B][chunk_tokens][d_model]
  const uint16_t* w_dkv;  // [d_c][d_model]
  const uint16_t* w_kr;   // [d_rope][d_model]
  const uint16_t* gamma;  // [d_c] or nullptr
  uint16_t* c_kv;         // [B][ring_tokens][d_c]
  uint16_t* k_r;          // [B][ring_tokens][d_rope]
  int32_t* slots;         // [chunk_tokens] or nullptr
  const uint16_t* w_packed;  // packed [W_DKV; W_KR] panel (cache_write_packed_kernel), or nullptr
  uint16_t* w_packed_out;    // pack_write_weights_kernel output
  int32_t batch, d_model, d_c, d_rope;
  int32_t tok_per_wg;     // tokens of the flat [B][chunk] order per workgroup (1 .. 32)
  int32_t n_cu;           // compute units of the device (the batched write's grid)
  float eps;
  Geometry geo;
  RopeTable rope;
};

struct AttendArgs {
#ifdef VMLA_PHASE_STAMPS
  uint64_t* stamps = stamp_buffer();
#endif
  const uint16_t* q_nope;  // [B][Nq][H][d_nope]
  const uint16_t* q_r;     // [B][Nq][H][d_rope]
  const uint16_t* w_uk;    // [H*d_nope][d_c]
  const uint16_t* w_uv;    // [H*d_v][d_c]
  const uint16_t* c_kv;    // ring
  const uint16_t* k_r;     // ring
  uint16_t* out;           // [B][Nq][H][d_v]
  uint16_t* qcat;          // workspace: [B*Nq*H][dqk_pad] bf16
  float* o_part;           // workspace: [max_seg][B*Nq*H][d_c] fp32
  float* ml_part;          // workspace: [max_seg][B*Nq*H][2] fp32 (running max, sum)
  uint16_t* k_rot;         // workspace (sink only): [B][ring_tokens][d_rope], rotated window keys
  int32_t batch, n_heads, d_nope, d_rope, d_c, d_v, dqk_pad;
  int32_t n_valid;         // valid ring slots (prefix of the ring)
  // Work partition of the attention kernel: units are (batch, row block, key tile) triples in
  // that order; workgroup w processes units [w*U/G, (w+1)*U/G). A row block whose tiles are
  // spread over k workgroups leaves k partial results, in slots 0..k-1.
  int32_t n_wg;            // G
  int32_t att_rows;        // query rows per row block
  int32_t row_blocks;      // row blocks per batch element
  int32_t tiles_per_row;   // T = ceil(n_valid / keys per tile)
  int64_t units;           // U = batch * row_blocks * T
  int32_t max_seg;         // partial-result slots the workspace holds
  float qscale;            // softmax scale * log2(e), folded into the absorbed query
  // Weighted partition (optional): the state area of kBalSlot words in the workspace (see bal_*
  // below). bal_on: split by the weights the state holds (equal weights, i.e. the even split, if
  // it holds no valid record for this G); bal_rec: the call is adaptive, bal_prep_kernel has
  // set the weights from the previous adaptive call's times and the attention kernel records
  // its own. bal_on = 0: the even split above, the state is not read.
  uint32_t* bal_state;
  int32_t bal_on, bal_rec;
  Geometry geo;
  RopeTable rope;
  // dense per-head comparator only (rows are (head, token) pairs, each head padded to nq_pad)
  const uint16_t* q;       // [B][Nq][H][d_v] unrotated queries
  const uint16_t* kv;      // ring [B][ring_tokens][H][2 * d_v]: rotated K_h, then V_h
  int32_t nq_pad;          // query rows per head, a whole number of row blocks
};

// Dense comparator's cache write: K = W_K x (rotated by 3D RoPE over each whole head), V = W_V x.
struct DenseWriteArgs {
  const uint16_t* x;       // [B][chunk_tokens][d_model]
  const uint16_t* w_k;     // [H*d_v][d_model]
  const uint16_t* w_v;     // [H*d_v][d_model]
  uint16_t* kv;            // [B][ring_tokens][H][2 * d_v]
  int32_t* slots;          // [chunk_tokens] or nullptr
  int32_t batch, d_model, n_heads, d_head;
  Geometry geo;
  RopeTable rope;          // d_head / 2 pairs
};

// Plain bf16 GEMM out^T[o][token] = a[o][:] . b[token][:] (a [N][K], b [M][K], K % 64 == 0).
constexpr int kEpiStore = 0;  // out[token][o] (row stride ldo), bf16
constexpr int kEpiQcat = 1;   // q_cat rows (token, head): RMSNorm factor, RoPE, scale; see k_layer.hip
constexpr int kEpiHeads = 2;  // out[token][(o / head_w) head_ld + col_off + o % head_w], bf16, head_w % 8 == 0
struct GemmArgs {
  const uint16_t* a;       // [N][K] weight rows
  const uint16_t* b;       // [M][K] token rows
  uint16_t* out;
  int32_t M, N, K, ldo;
  int32_t epi;
  // q_cat epilogue: output column o = h (q_dc + q_dr) + c; row (token, h) of width ldo
  int32_t q_heads, q_dc, q_dr, q_norm_dim;
  // per-head epilogue: output column o goes to head o / head_w, column col_off + o % head_w
  int32_t head_w, head_ld, col_off;
  float qscale, eps;
  Geometry geo;            // token t of the flat [B][q_count] order is query t % q_count
  RopeTable rope;
};

// Packing of the whole layer's weights (see k_layer.hip).
struct PrepArgs {
  const uint16_t *w_dq, *gamma_q, *w_uq, *w_qr, *w_uk, *w_uv, *w_o;
  uint16_t *w_dq_pad, *wq_cat, *b_o;
  int32_t n_heads, d_model, d_nope, d_rope, d_c, d_v, d_q, d_q_pad, k_out_pad;
};

// Workgroup whose unit range [w*U/G, (w+1)*U/G) contains `unit`.
__host__ __device__ inline int attend_owner(int64_t unit, int64_t units, int n_wg) {
  return (int)(((unit + 1) * (int64_t)n_wg - 1) / units);
}

// Weighted partition of the attention units. Workgroup k runs on XCD k mod 8 and gets a share of
// the units proportional to its XCD's integer weight w[k mod 8] in [kBalMin, kBalMax]:
// workgroup k takes [start(k), start(k+1)) with start(k) = floor(U cum(k) / cum(G)), cum(k) the
// summed weights of workgroups 0 .. k-1. Equal weights give the even split. The state area holds
// the weights (words 0..7), the G they were set for (8), a marker (9) and each workgroup's
// duration in 100 MHz ticks (kBalHead + k) as the last adaptive call recorded it. An adaptive
// call first runs bal_prep_kernel (one workgroup, stream-ordered between the previous call's
// last reader of the weights and this call's attention kernel): it sets each XCD's weight
// proportional to the work per time that XCD achieved, writes G and the marker, and clears the
// durations. Any state that fails the checks means equal weights.
constexpr uint32_t kBalMin = 820, kBalMax = 1280, kBalOne = 1024, kBalMark = 0x564d4c42u;
constexpr int kBalHead = 16, kBalMaxWg = 4096, kBalSlot = kBalHead + kBalMaxWg;

// The weights a partition state holds for G workgroups: its words 0..7 if the marker, G and
// every weight check out, else equal weights.
__host__ __device__ inline void bal_weights(const uint32_t* st, int G, uint32_t (&w)[8]) {
  bool ok = st[9] == kBalMark && st[8] == (uint32_t)G;
  for (int x = 0; x < 8; ++x) ok = ok && st[x] >= kBalMin && st[x] <= kBalMax;
  for (int x = 0; x < 8; ++x) w[x] = ok ? st[x] : kBalOne;
}

__host__ __device__ inline int64_t bal_cum(const uint32_t* w, int k) {
  int64_t s = 0;
  for (int x = 0; x < 8; ++x) s += (int64_t)w[x] * (k > x ? (k - x + 7) / 8 : 0);
  return s;
}
__host__ __device__ inline int64_t bal_start(const uint32_t* w, int G, int64_t U, int k) {
  return U * bal_cum(w, k) / bal_cum(w, G);
}
// The workgroup whose range contains `unit`: the largest k < G with start(k) <= unit, i.e.
// with cum(k) <= C = floor(((unit + 1) cum(G) - 1) / U); cum(8q + j) = q S + w[0] + .. + w[j-1]
// with S the sum of the 8 weights, so k = 8 (C / S) + the number of leading weights whose sum
// stays within C mod S.
__host__ __device__ inline int bal_owner(const uint32_t* w, int G, int64_t U, int64_t unit) {
  const int64_t C = ((unit + 1) * bal_cum(w, G) - 1) / U;
  int64_t S = 0;
  for (int x = 0; x < 8; ++x) S += w[x];
  int64_t r = C % S, k = C / S * 8;
  for (int x = 0; x < 7 && r >= (int64_t)w[x]; ++x) {
    r -= w[x];
    ++k;
  }
  return (int)(k < G - 1 ? k : G - 1);
}
// floor(n / d) for n >= 0, d >= 1, exactly. Below 2^53 both operands are exact doubles, and
// the truncated, correctly rounded quotient is already floor(n / d): a quotient q + r/d with
// r >= 1 sits at least 1/d above q and 1/d below q + 1, more than half an ulp of it (at most
// n 2^-53 / d). The two correction steps only guard against a division that is not correctly
// rounded.
__host__ __device__ inline int64_t floor_div(int64_t n, int64_t d) {
  if (n >= (int64_t(1) << 53)) return n / d;
  int64_t q = (int64_t)((double)n / (double)d);
  if (q * d > n) --q;
  else if ((q + 1) * d <= n) ++q;
  return q;
}
// attend_owner and bal_owner with their divisions done by floor_div: the same results. The
// merge kernels compute a row block's split count per thread, where the 64-bit integer
// division sequence would dominate; the attention kernel keeps the integer forms, whose code
// its register allocation was tuned with.
__host__ __device__ inline int attend_owner_fd(int64_t unit, int64_t units, int n_wg) {
  return (int)floor_div((unit + 1) * (int64_t)n_wg - 1, units);
}
__host__ __device__ inline int bal_owner_fd(const uint32_t* w, int G, int64_t U, int64_t unit) {
  // C <= cum(G) <= kBalMax G < 2^32 for the at most 2^20 workgroups of a call; S < 2^14
  const uint32_t C = (uint32_t)floor_div((unit + 1) * bal_cum(w, G) - 1, U);
  uint32_t S = 0;
  for (int x = 0; x < 8; ++x) S += w[x];
  int64_t r = C % S, k = (int64_t)(C / S) * 8;
  for (int x = 0; x < 7 && r >= (int64_t)w[x]; ++x) {
    r -= w[x];
    ++k;
  }
  return (int)(k < G - 1 ? k : G - 1);
}

// Partial-result slots a row block of T units can need under any weights: every range holds at
// least floor(U kBalMin / (kBalMin + (G - 1) kBalMax)) - 1 units.
__host__ __device__ inline int bal_max_seg(int G, int64_t U, int T) {
  const int64_t min_len = U * kBalMin / (kBalMin + (int64_t)(G - 1) * kBalMax) - 1;
  if (min_len < 1) return G + 1;  // some range could be empty: never adaptive
  const int64_t n = (T + min_len - 1) / min_len + 1;
  return (int)(n < G ? n : G);
}

// Sets the calling thread's last-error message (videomla_last_error) and returns `code`; for
// the C-ABI sources other than videomla_api.cpp.
int report_error(int code, const char* fmt, ...);

// Launchers (one per kernel). Return the launch status.
hipError_t launch_cache_write(const WriteArgs& a, hipStream_t s);
int cache_write_tokens_per_wg(int64_t tokens, int n_cu);
hipError_t launch_pack_write_weights(const WriteArgs& a, hipStream_t s);
size_t write_weights_packed_elems(int d_model, int d_c, int d_rope);
hipError_t launch_q_absorb(const AttendArgs& a, hipStream_t s);
hipError_t launch_rope_window(const AttendArgs& a, hipStream_t s);
hipError_t launch_bal_prep(const AttendArgs& a, hipStream_t s);
hipError_t launch_latent_attend(const AttendArgs& a, hipStream_t s);
// out_proj of a call whose row blocks can be split over more workgroups than its in-kernel
// merge table holds (few-query calls): latent_merge first writes the merged bf16 o_lat rows
// [row][d_c] into the q_cat area (ld_olat = n_heads * d_c), which out_proj then reads.
bool out_proj_premerged(const AttendArgs& a);
hipError_t launch_out_proj(const AttendArgs& a, hipStream_t s);
hipError_t launch_dense_cache_write(const DenseWriteArgs& a, hipStream_t s);
hipError_t launch_dense_q_prep(const AttendArgs& a, hipStream_t s);
hipError_t launch_dense_attend(const AttendArgs& a, hipStream_t s);
hipError_t launch_dense_merge(const AttendArgs& a, hipStream_t s);
hipError_t launch_mat_q_prep(const AttendArgs& a, hipStream_t s);
hipError_t launch_mat_attend(const AttendArgs& a, hipStream_t s);
bool mat_attend_supported(int d_k, int d_v);
hipError_t launch_mat_rope_fill(const AttendArgs& a, uint16_t* kv, hipStream_t s);
hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s);
hipError_t launch_latent_merge(const AttendArgs& a, uint16_t* o_lat, int ld_olat, hipStream_t s);
hipError_t launch_prepare_weights(const PrepArgs& a, hipStream_t s);

// Shapes the attention kernel is instantiated for.
bool latent_attend_supported(int d_c, int d_rope);
size_t q_absorb_lds_bytes(int d_c, int d_rope, int d_nope);
int latent_attend_rows_per_block(int d_c, int d_rope);
int latent_attend_keys_per_tile(int d_c, int d_rope);
int latent_attend_wgs_per_cu(int d_c, int d_rope);
bool dense_attend_supported(int d_head);
int dense_attend_rows_per_block();
int dense_attend_keys_per_tile();

}  // namespace vmla
