// Device-side helpers for gfx950 (CDNA4): vector types, MFMA wrappers, bf16 conversion,
// LDS transpose reads, cross-half-wave exchange and the 3D-RoPE angle.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "vmla_internal.h"

namespace vmla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// D(32x32) += A(32x16) B(16x32). Lane l holds A[l%32][8(l/32) .. +8], B[8(l/32) .. +8][l%32];
// accumulator element 4i+j of lane l is D[8i + 4(l/32) + j][l%32].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ u32x4 as_u32x4(bf16x8 v) { return __builtin_bit_cast(u32x4, v); }

__device__ __forceinline__ u32x4 ldg16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ void stg16(uint16_t* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Round-to-nearest-even fp32 -> bf16 (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16x8 to_bf16x8(f32x8 v) { return __builtin_convertvector(v, bf16x8); }
__device__ __forceinline__ bf16x4 to_bf16x4(f32x4 v) { return __builtin_convertvector(v, bf16x4); }
__device__ __forceinline__ uint16_t to_bf16_bits(float v) {
  return __builtin_bit_cast(uint16_t, (__bf16)v);
}
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

typedef __attribute__((address_space(3))) uint16_t lds_u16;

// Pointer into LDS in the LDS address space (so that constant offsets fold into the
// instruction's immediate offset).
__device__ __forceinline__ const lds_u16* as_lds(const uint16_t* p) {
  return (const lds_u16*)(p);
}

typedef __attribute__((address_space(3))) void lds_void;

// Direct global-to-LDS load of 16 B per lane: lane l's bytes land at LDS address lds_base + 16 l.
// Issued as inline assembly so that the compiler does not treat it as an LDS write it must wait
// for before every LDS read and barrier; the callers order it with explicit vmcnt waits (the
// load counts as one outstanding vector-memory operation until its data is in LDS).
__device__ __forceinline__ void lds_dma16(const uint16_t* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(lds_void*)(p);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int VM>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Phase stamps (diagnostic build only; see vmla_internal.h). VMLA_STAMP(args, kernel, point)
// records the real-time counter for this (workgroup, wave) with a plain vector store from lane 0;
// VMLA_STAMP_DRAINED first waits for the wave's outstanding memory operations, so that the
// point marks their completion. VMLA_STAMP_NOW() reads the counter only, and
// VMLA_STAMP_AT(args, kernel, point, t) stores such a reading later, where the store cannot
// delay a wait that follows the point. All are fenced for the scheduler, so that the point
// stays where it is written. In the product build they are empty (VMLA_STAMP_NOW() is 0).
#ifdef VMLA_PHASE_STAMPS
__device__ __forceinline__ uint64_t stamp_now() {
  __builtin_amdgcn_sched_barrier(0);
  const uint64_t now = __builtin_amdgcn_s_memrealtime();
  __builtin_amdgcn_sched_barrier(0);
  return now;
}
__device__ __forceinline__ void phase_stamp_at(uint64_t* buf, int kernel, int point, uint64_t t) {
  const int wg = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  const int wave = threadIdx.x >> 6;  // every stamped kernel has one-dimensional workgroups
  if (buf != nullptr && (threadIdx.x & 63) == 0 && wg < kStampWorkgroups && wave < kStampWaves)
    buf[(((int64_t)kernel * kStampWorkgroups + wg) * kStampWaves + wave) * kStampPoints + point] = t;
  __builtin_amdgcn_sched_barrier(0);
}
#define VMLA_STAMP_NOW() ::vmla::stamp_now()
#define VMLA_STAMP_AT(args, kernel, point, t) ::vmla::phase_stamp_at((args).stamps, (kernel), (point), (t))
#define VMLA_STAMP(args, kernel, point) VMLA_STAMP_AT(args, kernel, point, ::vmla::stamp_now())
#define VMLA_STAMP_DRAINED(args, kernel, point) \
  do {                                          \
    ::vmla::wait_vmcnt<0>();                    \
    VMLA_STAMP(args, kernel, point);            \
  } while (0)
#else
#define VMLA_STAMP_NOW() ((uint64_t)0)
#define VMLA_STAMP_AT(args, kernel, point, t) ((void)0)
#define VMLA_STAMP(args, kernel, point) ((void)0)
#define VMLA_STAMP_DRAINED(args, kernel, point) ((void)0)
#endif

// LDS transpose read (ds_read_b64_tr_b16). Within each group of 16 lanes, source lane s points
// at 4 consecutive 16-bit elements M[s][0..3]; result lane i receives M[4e + i/4][i%4],
// e = 0..3. If source lane s addresses row (R0 + s/4), columns C0 + 4(s%4) .. +4 of a row-major
// matrix, lane i receives column C0 + i of rows R0 .. R0+3.
__device__ __forceinline__ i16x4 lds_read_tr(const lds_u16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
}
__device__ __forceinline__ i16x4 lds_read_tr(const uint16_t* p) { return lds_read_tr(as_lds(p)); }

__device__ __forceinline__ bf16x8 join_bf16x8(i16x4 lo, i16x4 hi) {
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// Value of lane l ^ 32 (v_permlane32_swap): the swap returns {own-or-partner} pairs whose two
// entries are, on every lane, this lane's value and its partner's.
__device__ __forceinline__ float half_swap_max(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr bf16x2 kOnesBf16x2 = {(__bf16)1.0f, (__bf16)1.0f};

// Absolute position of chunk token n: (f, y, x).
struct TokenPos {
  int64_t f;
  int32_t y, x;
};
__device__ __forceinline__ TokenPos token_pos(const Geometry& g, int n) {
  const int hw = g.grid_h * g.grid_w;
  TokenPos p;
  p.f = g.frame_end + n / hw;
  const int r = n % hw;
  p.y = r / g.grid_w;
  p.x = r % g.grid_w;
  return p;
}
// Absolute position of query token n of an attention call (chunk token q_begin + n).
__device__ __forceinline__ TokenPos query_pos(const Geometry& g, int n) {
  return token_pos(g, g.q_begin + n);
}
// Frame slot of absolute frame f: f mod W without a sink; with S sink frames, f for f < S and
// S + (f - S) mod (W - S) otherwise.
__device__ __forceinline__ int64_t frame_slot(const Geometry& g, int64_t f) {
  const int S = g.sink_frames;
  return f < S ? f : S + (f - S) % (g.window_frames - S);
}
__device__ __forceinline__ int64_t ring_slot(const Geometry& g, const TokenPos& p) {
  return (frame_slot(g, p.f) * g.grid_h + p.y) * (int64_t)g.grid_w + p.x;
}
// Position a query of the chunk is rotated at: absolute without a sink, window-local with one.
__device__ __forceinline__ TokenPos rope_pos(const Geometry& g, TokenPos p) {
  if (g.sink_frames > 0 && p.f >= g.sink_frames) p.f = g.sink_frames + (p.f - g.local_lo);
  return p;
}

// One RoPE pair's axis and frequency, read from the table once (the table sits in the kernel
// arguments: with a per-lane pair index every read is a vector load that waits for all loads in
// flight, so loops whose lanes keep one pair read it before they start).
struct RopePair {
  int axis;
  double theta;
};
__device__ __forceinline__ RopePair rope_pair(const RopeTable& t, int pair) {
  return RopePair{t.axis[pair], t.theta[pair]};
}

// (cos, sin) of the pair's angle pos_axis * theta at position p: the angle in turns is reduced
// to [-1/2, 1/2] in double precision (pos * theta / 2pi minus its nearest integer), and the
// hardware cosine and sine, which take their argument in turns, finish it. Over that range they
// are within 1.3e-7 (2^-22.9) of the exact values, measured against double precision on 2^22
// points; the library sincosf of the angle in radians, whose fp32 product 2 pi r rounds first,
// is within 2.1e-7. Either is far below the bf16 rounding of the rotated vectors.
__device__ __forceinline__ f32x2 rope_cos_sin_at(double pos, double theta) {
  const double turns = pos * theta * 0.15915494309189533577;  // 1 / (2 pi)
  const float r = (float)(turns - rint(turns));
  return f32x2{__builtin_amdgcn_cosf(r), __builtin_amdgcn_sinf(r)};
}
// The position along the pair's axis (0: frame, 1: row, 2: column).
__device__ __forceinline__ double rope_axis_pos(int axis, const TokenPos& p) {
  return axis == 0 ? (double)p.f : (axis == 1 ? (double)p.y : (double)p.x);
}
__device__ __forceinline__ f32x2 rope_cos_sin(const RopePair& rp, const TokenPos& p) {
  return rope_cos_sin_at(rope_axis_pos(rp.axis, p), rp.theta);
}
__device__ __forceinline__ f32x2 rope_cos_sin(const RopeTable& t, int pair, const TokenPos& p) {
  return rope_cos_sin(rope_pair(t, pair), p);
}

// Rotate (u, v) by a (cos, sin) pair: (u cos - v sin, u sin + v cos) in fp32.
__device__ __forceinline__ void rotate_by(f32x2 cs, float& u, float& v) {
  const float ru = u * cs[0] - v * cs[1];
  const float rv = u * cs[1] + v * cs[0];
  u = ru;
  v = rv;
}

// Rotate the pair (u, v) of RoPE pair `pair` at position p by its angle pos_axis * theta.
__device__ __forceinline__ void rope_rotate(const RopeTable& t, int pair, const TokenPos& p,
                                            float& u, float& v) {
  rotate_by(rope_cos_sin(t, pair, p), u, v);
}

// Partial results of row block rbg: the workgroups owning its first and last units, under the
// even split or (bal_on) the weighted one whose weights the partition state holds (unchanged
// since the attention kernel read them: only bal_prep_kernel writes them, before it).
__device__ inline int attend_split_count(const AttendArgs& a, int64_t rbg) {
  const int64_t lo = rbg * a.tiles_per_row, hi = lo + a.tiles_per_row - 1;
  if (!a.bal_on) return attend_owner_fd(hi, a.units, a.n_wg) - attend_owner_fd(lo, a.units, a.n_wg) + 1;
  uint32_t w[8];
  bal_weights(a.bal_state, a.n_wg, w);
  return bal_owner_fd(w, a.n_wg, a.units, hi) - bal_owner_fd(w, a.n_wg, a.units, lo) + 1;
}

}  // namespace vmla
