// C-ABI layer: argument validation, ring/window arithmetic, workspace carving, dispatch of the
// kernels and optional per-kernel HIP-event timing. All checks run on the host before any
// launch, so every error path is reachable without a GPU.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "videomla.h"
#ifdef VMLA_PHASE_STAMPS
#include "videomla_stamps.h"
#endif
#include "vmla_internal.h"

using namespace vmla;

namespace {

thread_local std::string g_err;

void set_error(const char* fmt, va_list ap) {
  char buf[512];
  vsnprintf(buf, sizeof buf, fmt, ap);
  g_err = buf;
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  set_error(fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err.clear();
  return VIDEOMLA_OK;
}

}  // namespace

int vmla::report_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  set_error(fmt, ap);
  va_end(ap);
  return code;
}

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Shape checks common to every call.
int check_dims(const videomla_dims* d) {
  if (!d) return fail(VIDEOMLA_EINVAL, "dims is NULL");
  if (d->d_model <= 0 || d->n_heads <= 0 || d->d_nope <= 0 || d->d_rope <= 0 || d->d_c <= 0 ||
      d->d_v <= 0 || d->grid_h <= 0 || d->grid_w <= 0 || d->window_frames <= 0 ||
      d->chunk_frames <= 0)
    return fail(VIDEOMLA_EINVAL, "all sizes in dims must be positive");
  if (d->d_rope % 2) return fail(VIDEOMLA_EINVAL, "d_rope must be even (complex pairs), got %d", d->d_rope);
  if (d->rope_pairs[0] < 0 || d->rope_pairs[1] < 0 || d->rope_pairs[2] < 0 ||
      2 * (d->rope_pairs[0] + d->rope_pairs[1] + d->rope_pairs[2]) != d->d_rope)
    return fail(VIDEOMLA_EINVAL, "rope_pairs (%d,%d,%d) must be non-negative and sum to d_rope/2 = %d",
                d->rope_pairs[0], d->rope_pairs[1], d->rope_pairs[2], d->d_rope / 2);
  for (int a = 0; a < 3; ++a)
    if (d->rope_band_dim[a] < 0) return fail(VIDEOMLA_EINVAL, "rope_band_dim must be >= 0");
  if (!(d->rope_base > 0.f)) return fail(VIDEOMLA_EINVAL, "rope_base must be positive");
  if (!(d->softmax_scale >= 0.f)) return fail(VIDEOMLA_EINVAL, "softmax_scale must be >= 0");
  if (!(d->kv_norm_eps >= 0.f)) return fail(VIDEOMLA_EINVAL, "kv_norm_eps must be >= 0");
  if (d->chunk_frames > d->window_frames)
    return fail(VIDEOMLA_EINVAL, "chunk_frames (%d) exceeds window_frames (%d)", d->chunk_frames,
                d->window_frames);
  if (d->sink_frames < 0 || d->window_frames - d->sink_frames < d->chunk_frames)
    return fail(VIDEOMLA_EINVAL,
                "sink_frames (%d) must be >= 0 and leave a whole chunk (%d frames) of the %d-frame window",
                d->sink_frames, d->chunk_frames, d->window_frames);
  const int64_t ring = (int64_t)d->window_frames * d->grid_h * d->grid_w;
  if (ring > (int64_t)1 << 30) return fail(VIDEOMLA_EUNSUPPORTED, "ring of %lld tokens is too large", (long long)ring);
  if (d->d_rope / 2 > kMaxRopePairs) return fail(VIDEOMLA_EUNSUPPORTED, "d_rope > %d", 2 * kMaxRopePairs);
  return VIDEOMLA_OK;
}

int check_window(const videomla_window* w) {
  if (!w) return fail(VIDEOMLA_EINVAL, "window is NULL");
  if (w->frame_end < 0) return fail(VIDEOMLA_EINVAL, "frame_end must be >= 0, got %lld", (long long)w->frame_end);
  return VIDEOMLA_OK;
}

RopeTable make_rope(const videomla_dims* d) {
  RopeTable t{};
  t.n_pairs = d->d_rope / 2;
  int p = 0;
  for (int a = 0; a < 3; ++a) {
    const int n = d->rope_pairs[a];
    const double band = d->rope_band_dim[a] > 0 ? d->rope_band_dim[a] : 2.0 * n;
    for (int k = 0; k < n; ++k, ++p) {
      t.axis[p] = a;
      t.theta[p] = std::pow((double)d->rope_base, -2.0 * k / band);
    }
  }
  return t;
}

Geometry make_geo(const videomla_dims* d, const videomla_window* w) {
  Geometry g{};
  g.grid_h = d->grid_h;
  g.grid_w = d->grid_w;
  g.window_frames = d->window_frames;
  g.chunk_tokens = d->chunk_frames * d->grid_h * d->grid_w;
  g.q_begin = 0;
  g.q_count = g.chunk_tokens;
  g.frame_end = w->frame_end;
  g.ring_tokens = (int64_t)d->window_frames * d->grid_h * d->grid_w;
  g.sink_frames = d->sink_frames;
  if (d->sink_frames > 0) {  // first recent frame of the context: max(S, hi - (W - S))
    const int64_t hi = w->frame_end + d->chunk_frames;
    const int64_t lo = hi - (d->window_frames - d->sink_frames);
    g.local_lo = lo > d->sink_frames ? lo : d->sink_frames;
  }
  return g;
}

}  // namespace

// ---- timing ---------------------------------------------------------------------------------
// A caller-owned timer: the event pairs of the launches it bracketed, not yet read, and a pool of
// events to reuse. Used by one thread at a time.
struct videomla_timer {
  struct Rec {
    int kernel;
    hipEvent_t start, stop;
  };
  int only = -1;  // >= 0: time only this kernel
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  Rec open{-1, nullptr, nullptr};  // videomla_timer_begin without its end yet
};

namespace {

enum KernelId {
  K_Q_ABSORB = 0, K_LATENT_ATTEND, K_OUT_PROJ, K_ROPE_WINDOW, K_BAL_PREP,
  K_MAT_KV, K_MAT_Q_PREP, K_MAT_ATTEND, K_MAT_MERGE,
  K_DENSE_Q_PREP, K_DENSE_ATTEND, K_DENSE_MERGE,
  K_Q_DOWN, K_Q_UP, K_LATENT_MERGE, K_OUT_MIX, K_CACHE_WRITE, K_DENSE_CACHE_WRITE, K_COUNT
};
const char* kKernelNames[K_COUNT] = {"q_absorb",     "latent_attend", "out_proj",
                                     "rope_window",  "bal_prep",      "mat_kv",
                                     "mat_q_prep",   "mat_attend",    "mat_merge",
                                     "dense_q_prep", "dense_attend",  "dense_merge",
                                     "q_down",       "q_up",          "latent_merge",
                                     "out_mix",      "cache_write",   "dense_cache_write"};

int kernel_id(const char* name) {
  for (int k = 0; k < K_COUNT; ++k)
    if (std::strcmp(name, kKernelNames[k]) == 0) return k;
  return -1;
}

hipEvent_t take_event(videomla_timer* t) {
  if (!t->pool.empty()) {
    hipEvent_t e = t->pool.back();
    t->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  // timing only: GPU-side intervals on one device, so no system-scope fence (a lighter marker)
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

template <class F>
hipError_t timed(videomla_timer* t, int kernel, hipStream_t s, F&& launch) {
  if (!t || (t->only >= 0 && kernel != t->only)) return launch();
  hipEvent_t e0 = take_event(t), e1 = take_event(t);
  if (!e0 || !e1) {
    if (e0) t->pool.push_back(e0);
    if (e1) t->pool.push_back(e1);
    return launch();
  }
  if (hipEventRecord(e0, s) != hipSuccess) {
    t->pool.push_back(e0);
    t->pool.push_back(e1);
    return launch();
  }
  const hipError_t err = launch();
  if (hipEventRecord(e1, s) != hipSuccess) {
    t->pool.push_back(e0);
    t->pool.push_back(e1);
    return err;
  }
  t->pending.push_back({kernel, e0, e1});
  return err;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(VIDEOMLA_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
}

int device_cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
    return n;
  return 256;  // MI355X; used only when no device is visible (host-side size queries)
}

// ---- options ----------------------------------------------------------------------------------
// The options of one attention call, validated, with the query range resolved.
struct Opts {
  int n_wg;       // requested workgroups (0 = one per compute unit, or per resident slot)
  int partition;  // VIDEOMLA_PARTITION_*
  int form;       // VIDEOMLA_FORM_* (AUTO resolved by the caller)
  int q_begin, q_count;
  videomla_timer* timer;
};

int resolve_opts(const videomla_dims* d, const videomla_attend_opts* o, Opts& r) {
  const int chunk = d->chunk_frames * d->grid_h * d->grid_w;
  r = Opts{0, VIDEOMLA_PARTITION_EVEN, VIDEOMLA_FORM_LATENT, 0, chunk, nullptr};
  if (!o) return VIDEOMLA_OK;
  if (o->n_workgroups < 0 || o->n_workgroups > (1 << 20))
    return fail(VIDEOMLA_EINVAL, "n_workgroups must be in [0, 2^20], got %d", o->n_workgroups);
  if (o->partition < VIDEOMLA_PARTITION_EVEN || o->partition > VIDEOMLA_PARTITION_FROZEN)
    return fail(VIDEOMLA_EINVAL, "unknown partition mode %d", o->partition);
  if (o->form < VIDEOMLA_FORM_LATENT || o->form > VIDEOMLA_FORM_AUTO)
    return fail(VIDEOMLA_EINVAL, "unknown attention form %d", o->form);
  if (o->query_begin < 0 || o->query_begin >= chunk || o->query_count < 0 ||
      o->query_count > chunk - o->query_begin)
    return fail(VIDEOMLA_EINVAL, "query range [%d, %d + %d) outside the chunk's %d tokens",
                o->query_begin, o->query_begin, o->query_count, chunk);
  r.n_wg = o->n_workgroups;
  r.partition = o->partition;
  r.form = o->form;
  r.q_begin = o->query_begin;
  r.q_count = o->query_count > 0 ? o->query_count : chunk - o->query_begin;
  r.timer = o->timer;
  return VIDEOMLA_OK;
}

// ---- work partition ---------------------------------------------------------------------------
constexpr int kMaxSplitsPerRowBlock = 64;
// Work partition of the attention kernel for a window of n_valid keys (see AttendArgs).
struct Partition {
  int G, rows, RB, T, max_seg;
  int64_t U;
};

// rows: query rows per row block; RB: row blocks per batch element; bn: keys per tile;
// wpc: resident workgroups per compute unit; n_wg: requested workgroups (0 = wpc per CU).
Partition make_partition(int rows, int RB, int bn, int wpc, int32_t batch, int64_t n_valid,
                         int n_wg) {
  Partition p{};
  p.rows = rows;
  p.RB = RB;
  p.T = (int)((n_valid + bn - 1) / bn);
  p.U = (int64_t)batch * p.RB * p.T;
  // by default at most kMaxSplitsPerRowBlock - 1 workgroups per row block: few-query calls
  // (few row blocks, each split over many workgroups) then give each workgroup at least 1/63 of
  // a row block's key tiles, which bounds the partial results they write, and the merge reads,
  // relative to the keys they read
  int64_t G = n_wg > 0 ? n_wg : (int64_t)device_cu_count() * wpc;
  if (n_wg == 0 && G > (int64_t)(kMaxSplitsPerRowBlock - 1) * batch * RB)
    G = (int64_t)(kMaxSplitsPerRowBlock - 1) * batch * RB;
  p.G = (int)(G < p.U ? G : p.U);
  p.max_seg = 1;
  for (int64_t rbg = 0; rbg < (int64_t)batch * p.RB; ++rbg) {
    const int n = attend_owner(rbg * p.T + p.T - 1, p.U, p.G) - attend_owner(rbg * p.T, p.U, p.G) + 1;
    if (n > p.max_seg) p.max_seg = n;
  }
  return p;
}

Partition attend_partition(const videomla_dims* d, int32_t batch, int64_t n_valid, const Opts& o) {
  const int rows = latent_attend_rows_per_block(d->d_c, d->d_rope);
  const int64_t rows_b = (int64_t)o.q_count * d->n_heads;
  return make_partition(rows, (int)((rows_b + rows - 1) / rows),
                        latent_attend_keys_per_tile(d->d_c, d->d_rope),
                        latent_attend_wgs_per_cu(d->d_c, d->d_rope), batch, n_valid, o.n_wg);
}

// Per-head forms (the dense comparator and the materialized form): every head's query rows
// padded to whole row blocks.
int head_nq_pad(const Opts& o) {
  const int rows = dense_attend_rows_per_block();
  return (o.q_count + rows - 1) / rows * rows;
}

Partition head_partition(const videomla_dims* d, int32_t batch, int64_t n_valid, const Opts& o) {
  const int rows = dense_attend_rows_per_block();
  return make_partition(rows, d->n_heads * (head_nq_pad(o) / rows), dense_attend_keys_per_tile(),
                        1, batch, n_valid, o.n_wg);
}

// Partial-result slots the workspace must hold for any window this shape can attend over
// (chunk_frames up to window_frames valid frames).
int workspace_max_seg(const videomla_dims* d, int32_t batch, const Opts& o, bool per_head) {
  int m = 1;
  for (int f = d->chunk_frames; f <= d->window_frames; ++f) {
    const int64_t n_valid = (int64_t)f * d->grid_h * d->grid_w;
    const int s = (per_head ? head_partition(d, batch, n_valid, o)
                            : attend_partition(d, batch, n_valid, o)).max_seg;
    if (s > m) m = s;
  }
  return m;
}

// Workspace of the attention kernels: q rows [rows][q_width] bf16, the partial results
// [n_seg][rows][o_width] fp32 and (max, sum) pairs [n_seg][rows][2] fp32, the rotated window keys
// (latent form with a sink), then the partition state.
struct WorkspaceLayout {
  size_t qcat_off, opart_off, ml_off, krot_off, bal_off, total;
  int n_seg;  // partial-result slots
};

WorkspaceLayout make_layout(size_t base, size_t rows, size_t q_width, size_t o_width, int n_seg,
                            size_t krot_bytes) {
  WorkspaceLayout w{};
  w.qcat_off = base;
  w.opart_off = w.qcat_off + round_up(rows * q_width * 2, 256);
  w.ml_off = w.opart_off + round_up((size_t)n_seg * rows * o_width * 4, 256);
  w.krot_off = w.ml_off + round_up((size_t)n_seg * rows * 2 * 4, 256);
  w.bal_off = w.krot_off + round_up(krot_bytes, 256);
  w.total = w.bal_off + round_up((size_t)kBalSlot * 4, 256);
  w.n_seg = n_seg;
  return w;
}

WorkspaceLayout latent_layout(const videomla_dims* d, int32_t batch, const Opts& o) {
  const size_t rows = (size_t)batch * o.q_count * d->n_heads;
  const size_t krot = d->sink_frames > 0
                          ? (size_t)batch * d->window_frames * d->grid_h * d->grid_w * d->d_rope * 2
                          : 0;
  return make_layout(0, rows, round_up((size_t)d->d_c + d->d_rope, 16), d->d_c,
                     workspace_max_seg(d, batch, o, false), krot);
}

// Dense comparator: q rows [B][H][nq_pad][d_v].
WorkspaceLayout dense_layout(const videomla_dims* d, int32_t batch, const Opts& o) {
  const size_t rows = (size_t)batch * d->n_heads * head_nq_pad(o);
  return make_layout(0, rows, d->d_v, d->d_v, workspace_max_seg(d, batch, o, true), 0);
}

// Materialized form: the reconstructed rows [B][ring][H][d_k + d_v] (d_k = d_nope + d_rope),
// then per-head q rows [B][H][nq_pad][d_k] and the rest as for the dense comparator.
struct MatLayout {
  size_t kv_off;
  WorkspaceLayout att;
};
MatLayout mat_layout(const videomla_dims* d, int32_t batch, const Opts& o) {
  const size_t dk = (size_t)d->d_nope + d->d_rope;
  const size_t kv = (size_t)batch * d->window_frames * d->grid_h * d->grid_w * d->n_heads *
                    (dk + d->d_v) * 2;
  const size_t rows = (size_t)batch * d->n_heads * head_nq_pad(o);
  MatLayout m{};
  m.kv_off = 0;
  m.att = make_layout(round_up(kv, 256), rows, dk, d->d_v, workspace_max_seg(d, batch, o, true), 0);
  return m;
}

// The weighted partition for a call (adaptive or frozen): only where every range keeps at least
// one unit under any weights and the workspace holds the partial results such ranges can leave.
void set_balance(AttendArgs& a, const Partition& P, char* ws, const WorkspaceLayout& L,
                 const Opts& o) {
  a.bal_state = reinterpret_cast<uint32_t*>(ws + L.bal_off);
  a.bal_on = o.partition != VIDEOMLA_PARTITION_EVEN && P.G <= kBalMaxWg &&
             bal_max_seg(P.G, P.U, P.T) <= L.n_seg;
  a.bal_rec = a.bal_on && o.partition == VIDEOMLA_PARTITION_ADAPTIVE;
  if (a.bal_on) a.max_seg = L.n_seg;
}

// Full-head RoPE of the dense comparator: channels (d - 4 floor(d/6), 2 floor(d/6),
// 2 floor(d/6)) over (t, h, w), each axis' band width equal to its channel count.
RopeTable make_dense_rope(const videomla_dims* d) {
  videomla_dims hd = *d;
  const int k = d->d_v / 6;
  const int ch[3] = {d->d_v - 4 * k, 2 * k, 2 * k};
  hd.d_rope = d->d_v;
  for (int a = 0; a < 3; ++a) {
    hd.rope_pairs[a] = ch[a] / 2;
    hd.rope_band_dim[a] = ch[a];
  }
  return make_rope(&hd);
}

int check_dense_head(const videomla_dims* d) {
  if (d->d_v % 4 || d->d_v / 2 > kMaxRopePairs)
    return fail(VIDEOMLA_EUNSUPPORTED, "dense head width d_v must be a multiple of 4 and <= %d, got %d",
                2 * kMaxRopePairs, d->d_v);
  return VIDEOMLA_OK;
}

// Packed weights of the whole layer: W_down^Q [d_q_pad][d_model], the per-head query matrix
// [H (d_c + d_rope)][d_q_pad], B [d_model][k_out_pad]; zero padding to whole 64-column chunks.
struct LayerWeightsLayout {
  int d_q_pad, k_out_pad;
  size_t wdq_off, wq_off, bo_off, total;
};

LayerWeightsLayout layer_weights_layout(const videomla_dims* d, int32_t d_q) {
  LayerWeightsLayout L{};
  L.d_q_pad = (int)round_up((size_t)d_q, 64);
  L.k_out_pad = (int)round_up((size_t)d->n_heads * d->d_c, 64);
  L.wdq_off = 0;
  L.wq_off = round_up((size_t)L.d_q_pad * d->d_model * 2, 256);
  L.bo_off = L.wq_off + round_up((size_t)d->n_heads * (d->d_c + d->d_rope) * L.d_q_pad * 2, 256);
  L.total = L.bo_off + round_up((size_t)d->d_model * L.k_out_pad * 2, 256);
  return L;
}

int check_layer_shape(const videomla_dims* d, int32_t d_q) {
  if (d_q <= 0 || d_q > (1 << 16)) return fail(VIDEOMLA_EINVAL, "d_q must be in [1, 65536], got %d", d_q);
  if (d->d_model % 64)
    return fail(VIDEOMLA_EUNSUPPORTED, "d_model must be a multiple of 64, got %d", d->d_model);
  return VIDEOMLA_OK;
}

int check_attend_shape(const videomla_dims* d) {
  if (!latent_attend_supported(d->d_c, d->d_rope))
    return fail(VIDEOMLA_EUNSUPPORTED,
                "attention kernel is built for (d_c, d_rope) in {(64,32),(128,32),(192,32),"
                "(256,32),(512,32),(16,8)}, got (%d,%d)",
                d->d_c, d->d_rope);
  if (d->d_nope % 16 || d->d_nope > 128)
    return fail(VIDEOMLA_EUNSUPPORTED, "d_nope must be a multiple of 16 and <= 128, got %d", d->d_nope);
  if (d->d_v % 32 || d->d_v > 256)
    return fail(VIDEOMLA_EUNSUPPORTED, "d_v must be a multiple of 32 and <= 256, got %d", d->d_v);
  if (q_absorb_lds_bytes(d->d_c, d->d_rope, d->d_nope) > 64 * 1024)
    return fail(VIDEOMLA_EUNSUPPORTED, "d_nope %d too large for the query kernel", d->d_nope);
  return VIDEOMLA_OK;
}

}  // namespace

extern "C" {

const char* videomla_last_error(void) { return g_err.c_str(); }

size_t videomla_cache_bytes_per_token(const videomla_dims* d) {
  if (check_dims(d)) return 0;
  return 2 * ((size_t)d->d_c + d->d_rope);
}

int64_t videomla_valid_tokens(const videomla_dims* d, const videomla_window* w) {
  if (check_dims(d) || check_window(w)) return -1;
  const int64_t frames = w->frame_end + d->chunk_frames;
  const int64_t f = frames < d->window_frames ? frames : d->window_frames;
  return f * d->grid_h * d->grid_w;
}

int64_t videomla_slot_of(const videomla_dims* d, int64_t f, int32_t y, int32_t x) {
  if (check_dims(d)) return -1;
  if (f < 0 || y < 0 || y >= d->grid_h || x < 0 || x >= d->grid_w) {
    fail(VIDEOMLA_EINVAL, "position (%lld,%d,%d) outside the grid", (long long)f, y, x);
    return -1;
  }
  const int64_t S = d->sink_frames;
  const int64_t fs = f < S ? f : S + (f - S) % (d->window_frames - S);
  return (fs * d->grid_h + y) * (int64_t)d->grid_w + x;
}

int videomla_window_advance(const videomla_dims* d, videomla_window* w) {
  if (int e = check_dims(d)) return e;
  if (int e = check_window(w)) return e;
  w->frame_end += d->chunk_frames;
  return ok();
}

namespace {

// Shapes the cache-write kernels tile (shared by the plain and the packed-weight entry points).
int check_write_dims(const videomla_dims* d) {
  if (int e = check_dims(d)) return e;
  if (d->d_model % 64) return fail(VIDEOMLA_EUNSUPPORTED, "d_model must be a multiple of 64, got %d", d->d_model);
  if (d->d_model > kMaxWriteDModel)
    return fail(VIDEOMLA_EUNSUPPORTED, "d_model must be <= %d for the cache write, got %d", kMaxWriteDModel, d->d_model);
  if (d->d_c % 16) return fail(VIDEOMLA_EUNSUPPORTED, "d_c must be a multiple of 16, got %d", d->d_c);
  if (d->d_rope % 8) return fail(VIDEOMLA_EUNSUPPORTED, "d_rope must be a multiple of 8, got %d", d->d_rope);
  if (d->d_c + d->d_rope > kMaxWriteOutPacked)
    return fail(VIDEOMLA_EUNSUPPORTED, "d_c + d_rope must be <= %d", kMaxWriteOutPacked);
  return 0;
}

// Validation and launch common to videomla_cache_write (w_packed == NULL) and
// videomla_cache_write_prepared (w_dkv == w_kr == NULL).
int cache_write_common(const videomla_dims* d, const videomla_window* w, int32_t batch,
                       const uint16_t* x, const uint16_t* w_dkv, const uint16_t* w_kr,
                       const uint16_t* w_packed, const uint16_t* kv_norm_w, uint16_t* c_kv,
                       uint16_t* k_r, int32_t* slots_out, void* stream) {
  if (int e = check_write_dims(d)) return e;
  if (!w_packed && d->d_c + d->d_rope > kMaxWriteOutPlain)
    return fail(VIDEOMLA_EUNSUPPORTED,
                "d_c + d_rope must be <= %d for the plain-weight cache write (the packed-weight "
                "one takes up to %d)", kMaxWriteOutPlain, kMaxWriteOutPacked);
  if (int e = check_window(w)) return e;
  if (batch <= 0) return fail(VIDEOMLA_EINVAL, "batch must be positive, got %d", batch);
  if ((int64_t)batch * d->chunk_frames * d->grid_h * d->grid_w >= ((int64_t)1 << 31))
    return fail(VIDEOMLA_EUNSUPPORTED, "batch * chunk tokens must be < 2^31");
  if (!x || !c_kv || !k_r || (!w_packed && (!w_dkv || !w_kr)))
    return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  if (!aligned16(x) || !aligned16(c_kv) || !aligned16(k_r) ||
      (w_packed ? !aligned16(w_packed) : (!aligned16(w_dkv) || !aligned16(w_kr))))
    return fail(VIDEOMLA_EALIGN, "tensor pointers must be 16-byte aligned");
  if (kv_norm_w && !aligned16(kv_norm_w)) return fail(VIDEOMLA_EALIGN, "kv_norm_w must be 16-byte aligned");
  WriteArgs a{};
  a.x = x; a.w_dkv = w_dkv; a.w_kr = w_kr; a.w_packed = w_packed; a.gamma = kv_norm_w;
  a.c_kv = c_kv; a.k_r = k_r; a.slots = slots_out;
  a.batch = batch; a.d_model = d->d_model; a.d_c = d->d_c; a.d_rope = d->d_rope;
  a.eps = d->kv_norm_eps;
  a.geo = make_geo(d, w);
  a.rope = make_rope(d);
  a.n_cu = device_cu_count();
  a.tok_per_wg = cache_write_tokens_per_wg((int64_t)batch * a.geo.chunk_tokens, a.n_cu);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const hipError_t e = launch_cache_write(a, s);
  if (e != hipSuccess) return hip_fail(e, "cache_write");
  return ok();
}

}  // namespace

int videomla_cache_write(const videomla_dims* d, const videomla_window* w, int32_t batch,
                         const uint16_t* x, const uint16_t* w_dkv, const uint16_t* w_kr,
                         const uint16_t* kv_norm_w, uint16_t* c_kv, uint16_t* k_r,
                         int32_t* slots_out, void* stream) {
  if (!w_dkv || !w_kr) return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  return cache_write_common(d, w, batch, x, w_dkv, w_kr, nullptr, kv_norm_w, c_kv, k_r, slots_out,
                            stream);
}

size_t videomla_write_weights_bytes(const videomla_dims* d) {
  if (check_write_dims(d)) return 0;
  return write_weights_packed_elems(d->d_model, d->d_c, d->d_rope) * 2;
}

int videomla_prepare_write_weights(const videomla_dims* d, const uint16_t* w_dkv,
                                   const uint16_t* w_kr, uint16_t* w_packed, void* stream) {
  if (int e = check_write_dims(d)) return e;
  if (!w_dkv || !w_kr || !w_packed) return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  if (!aligned16(w_dkv) || !aligned16(w_kr) || !aligned16(w_packed))
    return fail(VIDEOMLA_EALIGN, "tensor pointers must be 16-byte aligned");
  WriteArgs a{};
  a.w_dkv = w_dkv; a.w_kr = w_kr; a.w_packed_out = w_packed;
  a.d_model = d->d_model; a.d_c = d->d_c; a.d_rope = d->d_rope;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const hipError_t e = launch_pack_write_weights(a, s);
  if (e != hipSuccess) return hip_fail(e, "prepare_write_weights");
  return ok();
}

int videomla_cache_write_prepared(const videomla_dims* d, const videomla_window* w, int32_t batch,
                                  const uint16_t* x, const uint16_t* w_packed,
                                  const uint16_t* kv_norm_w, uint16_t* c_kv, uint16_t* k_r,
                                  int32_t* slots_out, void* stream) {
  if (!w_packed) return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  return cache_write_common(d, w, batch, x, nullptr, nullptr, w_packed, kv_norm_w, c_kv, k_r,
                            slots_out, stream);
}

namespace {

// ---- attention ----------------------------------------------------------------------------------

int check_attend_args(const videomla_dims* d, const videomla_window* w, int32_t batch) {
  if (int e = check_dims(d)) return e;
  if (int e = check_window(w)) return e;
  if (batch <= 0) return fail(VIDEOMLA_EINVAL, "batch must be positive, got %d", batch);
  return VIDEOMLA_OK;
}

int check_workspace(const void* ws, size_t have, size_t need) {
  if (!ws || have < need)
    return fail(VIDEOMLA_EWORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                ws ? have : (size_t)0);
  if (!aligned16(ws)) return fail(VIDEOMLA_EALIGN, "workspace must be 16-byte aligned");
  return VIDEOMLA_OK;
}

// Materialized-K/V form: head rows [K_h | V_h] = [W_UK,h c ; k^R | W_UV,h c], keys of width
// d_nope + d_rope, values of width d_v; the attention kernel is built for 128 | 128 and 160 | 128.
bool materialized_supported(const videomla_dims* d) {
  return mat_attend_supported(d->d_nope + d->d_rope, d->d_v) && d->sink_frames == 0 &&
         d->d_c % 64 == 0 && d->d_rope % 8 == 0;
}

int check_materialized_shape(const videomla_dims* d) {
  if (!mat_attend_supported(d->d_nope + d->d_rope, d->d_v))
    return fail(VIDEOMLA_EUNSUPPORTED,
                "materialized attention is built for d_v = 128 and d_nope + d_rope in {128, 160}, "
                "got %d + %d, %d", d->d_nope, d->d_rope, d->d_v);
  if (d->sink_frames) return fail(VIDEOMLA_EUNSUPPORTED, "materialized attention has no sink mode");
  if (d->d_c % 64) return fail(VIDEOMLA_EUNSUPPORTED, "d_c must be a multiple of 64, got %d", d->d_c);
  if (d->d_rope % 8) return fail(VIDEOMLA_EUNSUPPORTED, "d_rope must be a multiple of 8, got %d", d->d_rope);
  return VIDEOMLA_OK;
}

// Cost model behind VIDEOMLA_FORM_AUTO, over a full window of S keys and R = batch x query
// tokens x heads query rows (each head's rows padded to whole row blocks in the materialized
// form, R_pad):
//   latent        kLatentFixed + R S (2 d_c + d_rope) / kLatentMacRate
//   materialized  kMatFixed + batch S H (d_k + d_v) 2 / kMatKvRate       (the reconstruction,
//                 bound by writing the rows) + R_pad S (d_k + d_v) / kMatMacRate
// with d_k = d_nope + d_rope; multiply-adds per score, bytes, seconds. The constants are a
// least-squares fit to the two forms' attend times measured on MI355X at the Wan geometry over
// d_nope 96 / 128, d_c 128 / 192 and 208, 1,560 and 4,680 query tokens (batch 1, 32,760 keys);
// with them the model picks the faster form at all twelve points.
constexpr double kLatentFixed = 67.8e-6;     // seconds: query absorption, merge, pipeline fill
constexpr double kLatentMacRate = 6.24e14;   // multiply-adds per second, latent attention
constexpr double kMatFixed = 56.3e-6;        // seconds: query preparation, merge, pipeline fill
constexpr double kMatKvRate = 2.45e12;       // bytes per second written by the reconstruction
constexpr double kMatMacRate = 5.56e14;      // multiply-adds per second, per-head attention

bool prefer_materialized(const videomla_dims* d, int32_t batch, const Opts& o) {
  if (!materialized_supported(d)) return false;
  const double S = (double)d->window_frames * d->grid_h * d->grid_w;
  const double R = (double)batch * o.q_count * d->n_heads;
  const double R_pad = (double)batch * head_nq_pad(o) * d->n_heads;
  const double dk = d->d_nope + d->d_rope;
  const double t_lat = kLatentFixed + R * S * (2.0 * d->d_c + d->d_rope) / kLatentMacRate;
  const double t_mat = kMatFixed + (double)batch * S * d->n_heads * (dk + d->d_v) * 2.0 / kMatKvRate +
                       R_pad * S * (dk + d->d_v) / kMatMacRate;
  return t_mat < t_lat;
}

// The form a videomla_attend_ex call runs (AUTO resolved); -1 with the error set if the options
// ask for the materialized form on a shape it is not built for.
int attend_form(const videomla_dims* d, int32_t batch, const Opts& o) {
  if (o.form == VIDEOMLA_FORM_MATERIALIZED) {
    if (check_materialized_shape(d)) return -1;
    return VIDEOMLA_FORM_MATERIALIZED;
  }
  if (o.form == VIDEOMLA_FORM_AUTO && prefer_materialized(d, batch, o))
    return VIDEOMLA_FORM_MATERIALIZED;
  return VIDEOMLA_FORM_LATENT;
}

// Attention arguments common to the latent form of videomla_attend_ex and videomla_attend_layer
// (shapes, window, query range, work partition, workspace carving); the caller sets the query
// and projection pointers.
AttendArgs attend_args(const videomla_dims* d, const videomla_window* w, int32_t batch,
                       const Opts& o, const WorkspaceLayout& L, char* ws, const uint16_t* c_kv,
                       const uint16_t* k_r) {
  AttendArgs a{};
  a.c_kv = c_kv; a.k_r = k_r;
  a.qcat = reinterpret_cast<uint16_t*>(ws + L.qcat_off);
  a.o_part = reinterpret_cast<float*>(ws + L.opart_off);
  a.ml_part = reinterpret_cast<float*>(ws + L.ml_off);
  a.k_rot = d->sink_frames > 0 ? reinterpret_cast<uint16_t*>(ws + L.krot_off) : nullptr;
  a.batch = batch; a.n_heads = d->n_heads; a.d_nope = d->d_nope; a.d_rope = d->d_rope;
  a.d_c = d->d_c; a.d_v = d->d_v;
  a.dqk_pad = (int32_t)round_up((size_t)d->d_c + d->d_rope, 16);
  a.geo = make_geo(d, w);
  a.geo.q_begin = o.q_begin;
  a.geo.q_count = o.q_count;
  a.rope = make_rope(d);
  a.n_valid = (int32_t)videomla_valid_tokens(d, w);
  const Partition P = attend_partition(d, batch, a.n_valid, o);
  a.n_wg = P.G;
  a.att_rows = P.rows;
  a.row_blocks = P.RB;
  a.tiles_per_row = P.T;
  a.units = P.U;
  a.max_seg = P.max_seg;
  set_balance(a, P, ws, L, o);
  const double scale = d->softmax_scale > 0.f ? (double)d->softmax_scale
                                              : 1.0 / std::sqrt((double)d->d_nope + d->d_rope);
  a.qscale = (float)(scale * 1.4426950408889634);
  return a;
}

// Arguments of the per-head forms (dense comparator: head width d_v, queries q; materialized:
// keys d_nope + d_rope wide). Rows are (head, token) pairs, each head padded to nq_pad.
AttendArgs head_args(const videomla_dims* d, const videomla_window* w, int32_t batch,
                     const Opts& o, const WorkspaceLayout& L, char* ws, bool materialized) {
  AttendArgs a{};
  a.qcat = reinterpret_cast<uint16_t*>(ws + L.qcat_off);
  a.o_part = reinterpret_cast<float*>(ws + L.opart_off);
  a.ml_part = reinterpret_cast<float*>(ws + L.ml_off);
  a.batch = batch; a.n_heads = d->n_heads; a.d_v = d->d_v; a.d_c = d->d_v;
  a.d_nope = materialized ? d->d_nope : 0;
  a.d_rope = materialized ? d->d_rope : 0;
  a.dqk_pad = materialized ? d->d_nope + d->d_rope : d->d_v;  // key width
  a.nq_pad = head_nq_pad(o);
  a.geo = make_geo(d, w);
  a.geo.q_begin = o.q_begin;
  a.geo.q_count = o.q_count;
  a.rope = materialized ? make_rope(d) : make_dense_rope(d);
  a.n_valid = (int32_t)videomla_valid_tokens(d, w);
  const Partition P = head_partition(d, batch, a.n_valid, o);
  a.n_wg = P.G;
  a.att_rows = P.rows;
  a.row_blocks = P.RB;
  a.tiles_per_row = P.T;
  a.units = P.U;
  a.max_seg = P.max_seg;
  set_balance(a, P, ws, L, o);
  const double dk = materialized ? (double)(d->d_nope + d->d_rope) : (double)d->d_v;
  const double scale = d->softmax_scale > 0.f ? (double)d->softmax_scale : 1.0 / std::sqrt(dk);
  a.qscale = (float)(scale * 1.4426950408889634);
  return a;
}

// The weights of an adaptive call (before its attention kernel), then the attention kernel.
int run_partition_prep(AttendArgs& a, videomla_timer* t, hipStream_t s) {
  if (!a.bal_rec) return VIDEOMLA_OK;
  const hipError_t e = timed(t, K_BAL_PREP, s, [&] { return launch_bal_prep(a, s); });
  if (e != hipSuccess) return hip_fail(e, "bal_prep");
  return VIDEOMLA_OK;
}

// The window keys at window-local time (sink only), the partition weights (adaptive only), then
// the attention kernel.
int run_attention(AttendArgs& a, videomla_timer* t, hipStream_t s) {
  hipError_t e;
  if (a.k_rot) {
    e = timed(t, K_ROPE_WINDOW, s, [&] { return launch_rope_window(a, s); });
    if (e != hipSuccess) return hip_fail(e, "rope_window");
    a.k_r = a.k_rot;
  }
  if (int r = run_partition_prep(a, t, s)) return r;
  e = timed(t, K_LATENT_ATTEND, s, [&] { return launch_latent_attend(a, s); });
  if (e != hipSuccess) return hip_fail(e, "latent_attend");
  return VIDEOMLA_OK;
}

// Workspace of a videomla_attend_ex call (0 with the error set when unsupported).
size_t attend_workspace(const videomla_dims* d, int32_t batch, const Opts& o, int form) {
  if (form == VIDEOMLA_FORM_MATERIALIZED) return mat_layout(d, batch, o).att.total;
  return latent_layout(d, batch, o).total;
}

int attend_impl(const videomla_dims* d, const videomla_window* w, int32_t batch,
                const uint16_t* q_nope, const uint16_t* q_r, const uint16_t* w_uk,
                const uint16_t* w_uv, const uint16_t* c_kv, const uint16_t* k_r, uint16_t* out,
                void* workspace, size_t workspace_bytes, const videomla_attend_opts* opts,
                void* stream) {
  if (int e = check_attend_args(d, w, batch)) return e;
  Opts o;
  if (int e = resolve_opts(d, opts, o)) return e;
  if (!q_nope || !q_r || !w_uk || !w_uv || !c_kv || !k_r || !out)
    return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  if (int e = check_attend_shape(d)) return e;
  const int form = attend_form(d, batch, o);
  if (form < 0) return VIDEOMLA_EUNSUPPORTED;
  if (!aligned16(q_nope) || !aligned16(q_r) || !aligned16(w_uk) || !aligned16(w_uv) ||
      !aligned16(c_kv) || !aligned16(k_r) || !aligned16(out))
    return fail(VIDEOMLA_EALIGN, "tensor pointers must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  videomla_timer* t = o.timer;

  if (form == VIDEOMLA_FORM_LATENT) {
    const WorkspaceLayout L = latent_layout(d, batch, o);
    if (int e = check_workspace(workspace, workspace_bytes, L.total)) return e;
    AttendArgs a = attend_args(d, w, batch, o, L, ws, c_kv, k_r);
    a.q_nope = q_nope; a.q_r = q_r; a.w_uk = w_uk; a.w_uv = w_uv; a.out = out;
    hipError_t e = timed(t, K_Q_ABSORB, s, [&] { return launch_q_absorb(a, s); });
    if (e != hipSuccess) return hip_fail(e, "q_absorb");
    if (int r = run_attention(a, t, s)) return r;
    if (out_proj_premerged(a)) {  // every row merged at once into the q_cat area, then W_UV
      e = timed(t, K_LATENT_MERGE, s, [&] {
        return launch_latent_merge(a, a.qcat, d->n_heads * d->d_c, s);
      });
      if (e != hipSuccess) return hip_fail(e, "latent_merge");
    }
    e = timed(t, K_OUT_PROJ, s, [&] { return launch_out_proj(a, s); });
    if (e != hipSuccess) return hip_fail(e, "out_proj");
    return ok();
  }

  // materialized: per-head K_h, V_h of every valid slot, then per-head attention
  const MatLayout M = mat_layout(d, batch, o);
  if (int e = check_workspace(workspace, workspace_bytes, M.att.total)) return e;
  uint16_t* kv = reinterpret_cast<uint16_t*>(ws + M.kv_off);
  AttendArgs a = head_args(d, w, batch, o, M.att, ws, true);
  a.q_nope = q_nope; a.q_r = q_r; a.k_r = k_r; a.kv = kv; a.out = out;
  const int64_t ring = a.geo.ring_tokens, H = d->n_heads, ld = (int64_t)a.dqk_pad + d->d_v;
  hipError_t e = timed(t, K_MAT_KV, s, [&] {
    // per batch element: K_h no-RoPE part = W_UK,h c and V_h = W_UV,h c of the valid slots
    for (int b = 0; b < batch; ++b) {
      GemmArgs g{};
      g.b = c_kv + (size_t)b * ring * d->d_c;
      g.out = kv + (size_t)b * ring * H * ld;
      g.M = a.n_valid; g.K = d->d_c; g.ldo = (int32_t)(H * ld); g.epi = kEpiHeads;
      g.head_ld = (int32_t)ld;
      g.a = w_uk; g.N = (int32_t)(H * d->d_nope); g.head_w = d->d_nope; g.col_off = 0;
      hipError_t r = launch_gemm_nt(g, s);
      if (r != hipSuccess) return r;
      g.a = w_uv; g.N = (int32_t)(H * d->d_v); g.head_w = d->d_v; g.col_off = a.dqk_pad;
      r = launch_gemm_nt(g, s);
      if (r != hipSuccess) return r;
    }
    return launch_mat_rope_fill(a, kv, s);
  });
  if (e != hipSuccess) return hip_fail(e, "mat_kv");
  e = timed(t, K_MAT_Q_PREP, s, [&] { return launch_mat_q_prep(a, s); });
  if (e != hipSuccess) return hip_fail(e, "mat_q_prep");
  if (int r = run_partition_prep(a, t, s)) return r;
  e = timed(t, K_MAT_ATTEND, s, [&] { return launch_mat_attend(a, s); });
  if (e != hipSuccess) return hip_fail(e, "mat_attend");
  e = timed(t, K_MAT_MERGE, s, [&] { return launch_dense_merge(a, s); });
  if (e != hipSuccess) return hip_fail(e, "mat_merge");
  return ok();
}

}  // namespace

size_t videomla_attend_workspace_bytes_ex(const videomla_dims* d, int32_t batch,
                                          const videomla_attend_opts* opts) {
  if (check_dims(d) || batch <= 0) return 0;
  Opts o;
  if (resolve_opts(d, opts, o)) return 0;
  if (check_attend_shape(d)) return 0;
  const int form = attend_form(d, batch, o);
  if (form < 0) return 0;
  return attend_workspace(d, batch, o, form);
}

size_t videomla_attend_workspace_bytes(const videomla_dims* d, int32_t batch) {
  return videomla_attend_workspace_bytes_ex(d, batch, nullptr);
}

int videomla_attend(const videomla_dims* d, const videomla_window* w, int32_t batch,
                    const uint16_t* q_nope, const uint16_t* q_r, const uint16_t* w_uk,
                    const uint16_t* w_uv, const uint16_t* c_kv, const uint16_t* k_r,
                    uint16_t* out, void* workspace, size_t workspace_bytes, void* stream) {
  return attend_impl(d, w, batch, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, workspace,
                     workspace_bytes, nullptr, stream);
}

int videomla_attend_ex(const videomla_dims* d, const videomla_window* w, int32_t batch,
                       const uint16_t* q_nope, const uint16_t* q_r, const uint16_t* w_uk,
                       const uint16_t* w_uv, const uint16_t* c_kv, const uint16_t* k_r,
                       uint16_t* out, void* workspace, size_t workspace_bytes,
                       const videomla_attend_opts* opts, void* stream) {
  return attend_impl(d, w, batch, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, workspace,
                     workspace_bytes, opts, stream);
}

// ---- dense comparator ---------------------------------------------------------------------------

size_t videomla_dense_cache_bytes_per_token(const videomla_dims* d) {
  if (check_dims(d)) return 0;
  return 2 * (size_t)d->n_heads * d->d_v * 2;
}

int videomla_dense_cache_write(const videomla_dims* d, const videomla_window* w, int32_t batch,
                               const uint16_t* x, const uint16_t* w_k, const uint16_t* w_v,
                               uint16_t* kv, int32_t* slots_out, void* stream) {
  if (int e = check_attend_args(d, w, batch)) return e;
  if (!x || !w_k || !w_v || !kv) return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  if (d->d_model % 64) return fail(VIDEOMLA_EUNSUPPORTED, "d_model must be a multiple of 64, got %d", d->d_model);
  if (int e = check_dense_head(d)) return e;
  if (d->sink_frames) return fail(VIDEOMLA_EUNSUPPORTED, "the dense comparator has no sink mode");
  if ((2 * d->n_heads * d->d_v) % 128)
    return fail(VIDEOMLA_EUNSUPPORTED, "2 * n_heads * d_v must be a multiple of 128, got %d",
                2 * d->n_heads * d->d_v);
  if (!aligned16(x) || !aligned16(w_k) || !aligned16(w_v) || !aligned16(kv))
    return fail(VIDEOMLA_EALIGN, "tensor pointers must be 16-byte aligned");
  DenseWriteArgs a{};
  a.x = x; a.w_k = w_k; a.w_v = w_v; a.kv = kv; a.slots = slots_out;
  a.batch = batch; a.d_model = d->d_model; a.n_heads = d->n_heads; a.d_head = d->d_v;
  a.geo = make_geo(d, w);
  a.rope = make_dense_rope(d);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const hipError_t e = launch_dense_cache_write(a, s);
  if (e != hipSuccess) return hip_fail(e, "dense_cache_write");
  return ok();
}

size_t videomla_dense_attend_workspace_bytes(const videomla_dims* d, int32_t batch,
                                             const videomla_attend_opts* opts) {
  if (check_dims(d) || batch <= 0) return 0;
  Opts o;
  if (resolve_opts(d, opts, o)) return 0;
  if (!dense_attend_supported(d->d_v)) return 0;
  return dense_layout(d, batch, o).total;
}

int videomla_dense_attend(const videomla_dims* d, const videomla_window* w, int32_t batch,
                          const uint16_t* q, const uint16_t* kv, uint16_t* out, void* workspace,
                          size_t workspace_bytes, const videomla_attend_opts* opts,
                          void* stream) {
  if (int e = check_attend_args(d, w, batch)) return e;
  Opts o;
  if (int e = resolve_opts(d, opts, o)) return e;
  if (!q || !kv || !out) return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  if (!dense_attend_supported(d->d_v))
    return fail(VIDEOMLA_EUNSUPPORTED, "dense attention is built for d_v = 128, got %d", d->d_v);
  if (d->sink_frames) return fail(VIDEOMLA_EUNSUPPORTED, "the dense comparator has no sink mode");
  if (!aligned16(q) || !aligned16(kv) || !aligned16(out))
    return fail(VIDEOMLA_EALIGN, "tensor pointers must be 16-byte aligned");
  const WorkspaceLayout L = dense_layout(d, batch, o);
  if (int e = check_workspace(workspace, workspace_bytes, L.total)) return e;

  AttendArgs a = head_args(d, w, batch, o, L, static_cast<char*>(workspace), false);
  a.q = q; a.kv = kv; a.out = out;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  videomla_timer* t = o.timer;
  hipError_t e = timed(t, K_DENSE_Q_PREP, s, [&] { return launch_dense_q_prep(a, s); });
  if (e != hipSuccess) return hip_fail(e, "dense_q_prep");
  if (int r = run_partition_prep(a, t, s)) return r;
  e = timed(t, K_DENSE_ATTEND, s, [&] { return launch_dense_attend(a, s); });
  if (e != hipSuccess) return hip_fail(e, "dense_attend");
  e = timed(t, K_DENSE_MERGE, s, [&] { return launch_dense_merge(a, s); });
  if (e != hipSuccess) return hip_fail(e, "dense_merge");
  return ok();
}

// ---- the whole attention layer ---------------------------------------------------------------

size_t videomla_layer_weights_bytes(const videomla_dims* d, int32_t d_q) {
  if (check_dims(d) || check_layer_shape(d, d_q)) return 0;
  return layer_weights_layout(d, d_q).total;
}

int videomla_prepare_layer_weights(const videomla_dims* d, int32_t d_q, const uint16_t* w_dq,
                                   const uint16_t* gamma_q, const uint16_t* w_uq,
                                   const uint16_t* w_qr, const uint16_t* w_uk,
                                   const uint16_t* w_uv, const uint16_t* w_o, void* weights,
                                   size_t weights_bytes, void* stream) {
  if (int e = check_dims(d)) return e;
  if (int e = check_layer_shape(d, d_q)) return e;
  if (!w_dq || !w_uq || !w_qr || !w_uk || !w_uv || !w_o || !weights)
    return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  const LayerWeightsLayout L = layer_weights_layout(d, d_q);
  if (weights_bytes < L.total)
    return fail(VIDEOMLA_EWORKSPACE, "layer weights need %zu bytes, %zu given", L.total, weights_bytes);
  if (!aligned16(weights)) return fail(VIDEOMLA_EALIGN, "weights must be 16-byte aligned");
  PrepArgs a{};
  a.w_dq = w_dq; a.gamma_q = gamma_q; a.w_uq = w_uq; a.w_qr = w_qr; a.w_uk = w_uk; a.w_uv = w_uv;
  a.w_o = w_o;
  char* base = static_cast<char*>(weights);
  a.w_dq_pad = reinterpret_cast<uint16_t*>(base + L.wdq_off);
  a.wq_cat = reinterpret_cast<uint16_t*>(base + L.wq_off);
  a.b_o = reinterpret_cast<uint16_t*>(base + L.bo_off);
  a.n_heads = d->n_heads; a.d_model = d->d_model; a.d_nope = d->d_nope; a.d_rope = d->d_rope;
  a.d_c = d->d_c; a.d_v = d->d_v; a.d_q = d_q; a.d_q_pad = L.d_q_pad; a.k_out_pad = L.k_out_pad;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const hipError_t e = launch_prepare_weights(a, s);
  if (e != hipSuccess) return hip_fail(e, "prepare_layer_weights");
  return ok();
}

namespace {
// attention workspace, then u = W_down^Q x [B q_count][d_q_pad] and o_lat [B q_count][k_out_pad],
// bf16
struct LayerWorkspace {
  WorkspaceLayout att;
  size_t u_off, olat_off, total;
};

LayerWorkspace layer_workspace(const videomla_dims* d, int32_t d_q, int32_t batch, const Opts& o) {
  const LayerWeightsLayout W = layer_weights_layout(d, d_q);
  LayerWorkspace L{};
  L.att = latent_layout(d, batch, o);
  const size_t tokens = (size_t)batch * o.q_count;
  L.u_off = L.att.total;
  L.olat_off = L.u_off + round_up(tokens * W.d_q_pad * 2, 256);
  L.total = L.olat_off + round_up(tokens * W.k_out_pad * 2, 256);
  return L;
}

int resolve_layer_opts(const videomla_dims* d, const videomla_attend_opts* opts, Opts& o) {
  if (int e = resolve_opts(d, opts, o)) return e;
  if (o.form == VIDEOMLA_FORM_MATERIALIZED)
    return fail(VIDEOMLA_EUNSUPPORTED, "the whole layer runs the latent form only");
  return VIDEOMLA_OK;
}
}  // namespace

size_t videomla_attend_layer_workspace_bytes(const videomla_dims* d, int32_t d_q, int32_t batch,
                                             const videomla_attend_opts* opts) {
  if (check_dims(d) || check_layer_shape(d, d_q) || batch <= 0) return 0;
  Opts o;
  if (resolve_layer_opts(d, opts, o)) return 0;
  if (!latent_attend_supported(d->d_c, d->d_rope)) return 0;
  return layer_workspace(d, d_q, batch, o).total;
}

int videomla_attend_layer(const videomla_dims* d, const videomla_window* w, int32_t batch,
                          int32_t d_q, const uint16_t* x, const void* weights,
                          size_t weights_bytes, const uint16_t* c_kv, const uint16_t* k_r,
                          uint16_t* y, void* workspace, size_t workspace_bytes,
                          const videomla_attend_opts* opts, void* stream) {
  if (int e = check_attend_args(d, w, batch)) return e;
  if (int e = check_layer_shape(d, d_q)) return e;
  Opts o;
  if (int e = resolve_layer_opts(d, opts, o)) return e;
  if (!x || !weights || !c_kv || !k_r || !y) return fail(VIDEOMLA_EINVAL, "NULL tensor pointer");
  if (int e = check_attend_shape(d)) return e;
  if (!aligned16(x) || !aligned16(weights) || !aligned16(c_kv) || !aligned16(k_r) || !aligned16(y))
    return fail(VIDEOMLA_EALIGN, "tensor pointers must be 16-byte aligned");
  const LayerWeightsLayout W = layer_weights_layout(d, d_q);
  if (weights_bytes < W.total)
    return fail(VIDEOMLA_EWORKSPACE, "layer weights of %zu bytes expected, %zu given", W.total,
                weights_bytes);
  const LayerWorkspace L = layer_workspace(d, d_q, batch, o);
  if (int e = check_workspace(workspace, workspace_bytes, L.total)) return e;

  char* ws = static_cast<char*>(workspace);
  const char* wb = static_cast<const char*>(weights);
  AttendArgs a = attend_args(d, w, batch, o, L.att, ws, c_kv, k_r);
  uint16_t* u = reinterpret_cast<uint16_t*>(ws + L.u_off);
  uint16_t* o_lat = reinterpret_cast<uint16_t*>(ws + L.olat_off);
  const int M = batch * o.q_count;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  videomla_timer* t = o.timer;

  GemmArgs g1{};  // u = W_down^Q x
  g1.a = reinterpret_cast<const uint16_t*>(wb + W.wdq_off); g1.b = x; g1.out = u;
  g1.M = M; g1.N = W.d_q_pad; g1.K = d->d_model; g1.ldo = W.d_q_pad; g1.epi = kEpiStore;
  hipError_t e = timed(t, K_Q_DOWN, s, [&] { return launch_gemm_nt(g1, s); });
  if (e != hipSuccess) return hip_fail(e, "q_down");

  GemmArgs g2{};  // q_cat from c^Q = g_Q u / rms(u) (the gain is in the packed weights)
  g2.a = reinterpret_cast<const uint16_t*>(wb + W.wq_off); g2.b = u; g2.out = a.qcat;
  g2.M = M; g2.N = d->n_heads * (d->d_c + d->d_rope); g2.K = W.d_q_pad; g2.ldo = a.dqk_pad;
  g2.epi = kEpiQcat;
  g2.q_heads = d->n_heads; g2.q_dc = d->d_c; g2.q_dr = d->d_rope; g2.q_norm_dim = d_q;
  g2.qscale = a.qscale; g2.eps = d->kv_norm_eps; g2.geo = a.geo; g2.rope = a.rope;
  e = timed(t, K_Q_UP, s, [&] { return launch_gemm_nt(g2, s); });
  if (e != hipSuccess) return hip_fail(e, "q_up");

  if (int r = run_attention(a, t, s)) return r;
  e = timed(t, K_LATENT_MERGE, s, [&] { return launch_latent_merge(a, o_lat, W.k_out_pad, s); });
  if (e != hipSuccess) return hip_fail(e, "latent_merge");

  GemmArgs g3{};  // y = [B_1 .. B_H] o_lat
  g3.a = reinterpret_cast<const uint16_t*>(wb + W.bo_off); g3.b = o_lat; g3.out = y;
  g3.M = M; g3.N = d->d_model; g3.K = W.k_out_pad; g3.ldo = d->d_model; g3.epi = kEpiStore;
  e = timed(t, K_OUT_MIX, s, [&] { return launch_gemm_nt(g3, s); });
  if (e != hipSuccess) return hip_fail(e, "out_mix");
  return ok();
}

// ---- timers -------------------------------------------------------------------------------------

int videomla_timer_create(videomla_timer** timer) {
  if (!timer) return fail(VIDEOMLA_EINVAL, "NULL timer pointer");
  *timer = new (std::nothrow) videomla_timer();
  if (!*timer) return fail(VIDEOMLA_EINVAL, "out of host memory");
  return ok();
}

int videomla_timer_destroy(videomla_timer* timer) {
  if (!timer) return ok();
  for (const auto& r : timer->pending) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  for (hipEvent_t e : timer->pool) (void)hipEventDestroy(e);
  if (timer->open.start) (void)hipEventDestroy(timer->open.start);
  delete timer;
  return ok();
}

int videomla_timer_only(videomla_timer* timer, const char* kernel) {
  if (!timer) return fail(VIDEOMLA_EINVAL, "NULL timer");
  if (!kernel) {
    timer->only = -1;
    return ok();
  }
  const int id = kernel_id(kernel);
  if (id < 0) return fail(VIDEOMLA_EINVAL, "unknown kernel name '%s'", kernel);
  timer->only = id;
  return ok();
}

int videomla_timer_begin(videomla_timer* timer, const char* kernel, void* stream) {
  if (!timer || !kernel) return fail(VIDEOMLA_EINVAL, "NULL argument");
  const int id = kernel_id(kernel);
  if (id < 0) return fail(VIDEOMLA_EINVAL, "unknown kernel name '%s'", kernel);
  if (timer->open.start) timer->pool.push_back(timer->open.start);  // an unmatched begin
  timer->open = {-1, nullptr, nullptr};
  hipEvent_t e = take_event(timer);
  if (!e) return fail(VIDEOMLA_EHIP, "hipEventCreate failed");
  const hipError_t r = hipEventRecord(e, reinterpret_cast<hipStream_t>(stream));
  if (r != hipSuccess) {
    timer->pool.push_back(e);
    return hip_fail(r, "hipEventRecord");
  }
  timer->open = {id, e, nullptr};
  return ok();
}

int videomla_timer_end(videomla_timer* timer, const char* kernel, void* stream) {
  if (!timer || !kernel) return fail(VIDEOMLA_EINVAL, "NULL argument");
  const int id = kernel_id(kernel);
  if (id < 0) return fail(VIDEOMLA_EINVAL, "unknown kernel name '%s'", kernel);
  if (!timer->open.start || timer->open.kernel != id)
    return fail(VIDEOMLA_EINVAL, "videomla_timer_end('%s') without its videomla_timer_begin", kernel);
  hipEvent_t e = take_event(timer);
  if (!e) return fail(VIDEOMLA_EHIP, "hipEventCreate failed");
  const hipError_t r = hipEventRecord(e, reinterpret_cast<hipStream_t>(stream));
  if (r != hipSuccess) {
    timer->pool.push_back(e);
    return hip_fail(r, "hipEventRecord");
  }
  timer->pending.push_back({id, timer->open.start, e});
  timer->open = {-1, nullptr, nullptr};
  return ok();
}

int videomla_timer_read(videomla_timer* timer, const char* kernel, int64_t* count,
                        double* total_ms) {
  if (!timer || !kernel || !count || !total_ms) return fail(VIDEOMLA_EINVAL, "NULL argument");
  const int id = kernel_id(kernel);
  if (id < 0) return fail(VIDEOMLA_EINVAL, "unknown kernel name '%s'", kernel);
  *count = 0;
  *total_ms = 0.0;
  std::vector<videomla_timer::Rec> keep;
  for (const auto& r : timer->pending) {
    if (r.kernel != id) {
      keep.push_back(r);
      continue;
    }
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      keep.push_back(r);
      continue;
    }
    *count += 1;
    *total_ms += ms;
    timer->pool.push_back(r.start);
    timer->pool.push_back(r.stop);
  }
  timer->pending.swap(keep);
  return ok();
}

}  // extern "C"

#ifdef VMLA_PHASE_STAMPS
// The diagnostic build's one process-wide setting: the buffer the next launches record into.
namespace {
uint64_t* g_stamps = nullptr;
static_assert(kStampBufferBytes == VIDEOMLA_STAMP_BUFFER_BYTES, "stamp buffer layout");
}  // namespace

uint64_t* vmla::stamp_buffer() { return g_stamps; }

extern "C" int videomla_stamps_attach(void* device_buffer, int64_t bytes) {
  if (device_buffer == nullptr) {
    g_stamps = nullptr;
    return ok();
  }
  if (bytes < kStampBufferBytes)
    return fail(VIDEOMLA_EINVAL, "stamp buffer of %lld bytes, %lld needed", (long long)bytes,
                (long long)kStampBufferBytes);
  if ((reinterpret_cast<uintptr_t>(device_buffer) & 7u) != 0)
    return fail(VIDEOMLA_EALIGN, "stamp buffer is not 8-byte aligned");
  g_stamps = static_cast<uint64_t*>(device_buffer);
  return ok();
}
#endif
