// Fused cache write: compress (Eq. 1), optional RMSNorm of the latent, decoupled RoPE key
// (Eq. 5) rotated at the token's absolute (f, y, x) (kept unrotated when the cache has an
// attention sink, Sec. "Decoupled 3D-RoPE"), and FIFO placement into the ring.
//
// The work is a skinny GEMM, out[token][o] = [W_DKV; W_KR][o][:] . x[token][:]: every token
// needs the whole weight panel (d_c + d_rope rows of d_model), each token row is needed once.
// Two kernels:
//
// cache_write_packed_kernel (weights packed once by pack_write_weights_kernel). A workgroup
// takes a block of at most 32 consecutive tokens of the flat [batch][chunk] order, sized so
// that the grid covers every CU once, and all outputs:
//   * the block's x rows are loaded into LDS once, up front, by direct global-to-LDS loads
//     (one memory latency, shared by all waves), in an XOR-swizzled layout that makes the
//     MFMA operand reads conflict-free;
//   * wave w owns outputs 32w .. 32w+31 and streams its slice of the packed panel from L2
//     straight into registers, several MFMA k-steps ahead of use. The panel is stored in
//     MFMA operand order, so each load reads 1 KB contiguous: full cache lines per
//     instruction, which the L1 path delivers about three times faster than the 16- or
//     32-row operand pattern read from the plain row-major weights;
//   * MFMA 16x16x32: A = 16 weight rows x 32 columns, B = 32 columns x 16 tokens;
//   * each workgroup starts its contraction at its own column offset, so that the
//     workgroups of one L2 do not all ask for the same weight lines at the same time.
//   The epilogue combines the RMSNorm sum of squares across waves in LDS, normalizes, rotates
//   the RoPE block, rounds to bf16 into an LDS tile, and stores every token's c_kv and k_r
//   rows whole (coalesced 16-byte stores) at its ring slot.
//
// cache_write_staged_kernel (plain row-major weights). One workgroup takes 32 chunk tokens and
// all outputs: out^T[o][token] = W[o][:] . x[token][:] with MFMA 32x32x16 (A = rows of
// [W_DKV; W_KR], B = x rows). The contraction over d_model streams through a ring of kStages
// LDS stages of kKC columns each, filled by direct global-to-LDS loads in an XOR-swizzled
// layout; the four waves share every staged chunk and split the 32-row output blocks between
// them. Same epilogue steps, with 8-byte stores straight from the accumulators.
#include <type_traits>

#include "vmla_device.h"

namespace vmla {
namespace {

constexpr int kTokTile = 32;   // token rows of the resident x tile: two 16-token MFMA blocks
constexpr int kMaxWaves = 9;   // d_c + d_rope <= 288 with 32 outputs per wave, 576 with 64

// D(16x16) += A(16x32) B(32x16). Lane l holds A[l%16][8(l/16) .. +8], B[8(l/16) .. +8][l%16];
// accumulator element i of lane l is D[4(l/16) + i][l%16].
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// RMSNorm sum of squares of token rows 16 tb + r (tb < TB): the sum over the waves w < n of
// part[w * stride + row], added in the order w = 0, 1, ... Every load is issued before the
// first add (rows of waves past n are read at wave n - 1 and replaced by zero, which leaves the
// sum unchanged); a loop bounded by the run-time n would wait for each load in turn.
template <int MAXW, int TB>
__device__ __forceinline__ void sum_wave_parts(const float* part, int stride, int n, int r,
                                               float (&tot)[TB]) {
  float v[MAXW][TB];
#pragma unroll
  for (int w = 0; w < MAXW; ++w) {
    const int wr = w < n ? w : n - 1;
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) v[w][tb] = part[wr * stride + 16 * tb + r];
  }
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    tot[tb] = 0.f;
#pragma unroll
    for (int w = 0; w < MAXW; ++w) tot[tb] += w < n ? v[w][tb] : 0.f;
  }
}

constexpr uint32_t kOneBf16x2 = 0x3F803F80u;  // two bf16 ones: the gain when there is none

// The epilogue's output tile: normalized latents times the gain, and rotated RoPE keys, rounded
// to bf16 into ot[t][0 .. NO) (row stride ots). Lane (r, q) holds outputs o0 + 16 ob + 4q + e
// (o0 = the wave's first output) of token 16 tb + r in acc[ob][tb][e]; gam[ob] holds the gains of
// its four latent outputs as bf16 pairs (ones without a gain), rstd[tb] the token's reciprocal
// RMS (one without a gain), rope_cs[t * cs_stride + i] the (cos, sin) of token t's pair i.
// With d_c % 16 == 0 every 16-output block is all latent or all RoPE key (and padding), so that
// the branch is uniform per block and the token blocks inside it are straight-line code, which
// the compiler interleaves; a per-lane branch inside the token loop would serialize them.
template <int OB, int TB>
__device__ __forceinline__ void write_out_tile(const f32x4 (&acc)[OB][TB], const u32x2 (&gam)[OB],
                                               const float (&rstd)[TB], const f32x2* rope_cs,
                                               int cs_stride, int o_wave, int DC, int NO, int r,
                                               int q, int ntok, uint16_t* ot, int ots) {
#pragma unroll
  for (int ob = 0; ob < OB; ++ob) {
    const int o0 = o_wave + 16 * ob;  // first output of the block
    const int o = o0 + 4 * q;         // first of this lane's four consecutive outputs
    if (o0 + 16 <= DC) {
      const float g0 = __uint_as_float(gam[ob][0] << 16);
      const float g1 = __uint_as_float(gam[ob][0] & 0xffff0000u);
      const float g2 = __uint_as_float(gam[ob][1] << 16);
      const float g3 = __uint_as_float(gam[ob][1] & 0xffff0000u);
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        f32x4 v = acc[ob][tb] * rstd[tb];
        v = f32x4{v[0] * g0, v[1] * g1, v[2] * g2, v[3] * g3};
        *reinterpret_cast<bf16x4*>(&ot[(16 * tb + r) * ots + o]) = to_bf16x4(v);
      }
    } else if (o0 < NO) {  // channels o-DC .. +3 = RoPE pairs (o-DC)/2 and (o-DC)/2 + 1
      const bool live = o < NO;  // else padding past d_c + d_rope
      const int pr = live ? (o - DC) / 2 : 0;
      // every (cos, sin) read before the first tile write: the compiler cannot tell the two LDS
      // areas apart, and would otherwise wait for each write before the next read
      f32x2 c0[TB], c1[TB];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const int t = 16 * tb + r;
        const int tc = t < ntok ? t : ntok - 1;
        c0[tb] = rope_cs[tc * cs_stride + pr];
        c1[tb] = rope_cs[tc * cs_stride + pr + 1];
      }
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const f32x4 v = acc[ob][tb];
        const f32x2 a0 = c0[tb], a1 = c1[tb];
        const f32x4 w = {v[0] * a0[0] - v[1] * a0[1], v[0] * a0[1] + v[1] * a0[0],
                         v[2] * a1[0] - v[3] * a1[1], v[2] * a1[1] + v[3] * a1[0]};
        if (live) *reinterpret_cast<bf16x4*>(&ot[(16 * tb + r) * ots + o]) = to_bf16x4(w);
      }
    }
  }
}

// x tile layout: column blocks of 64 columns (8 chunks of 16 bytes); block b holds rows
// 0 .. rows_pad-1 (rows_pad = the block's token count rounded up to 8) row-major, the chunk index
// XOR-ed with (row / 2) mod 8, so 16 rows read at one chunk hit 16 distinct 16-byte bank groups.
// A direct load fills 64 consecutive positions = 8 rows x 128 bytes of one block (whole lines).
__device__ __forceinline__ int xpos(int b, int t, int cc, int rows_pad) {
  return (b * rows_pad + t) * 8 + (cc ^ ((t >> 1) & 7));
}

// One wave per 16 OB outputs of d_c + d_rope (OB = 2, or 4 beyond 288 outputs). KPRE (weight
// k-steps of 32 columns in flight per wave) divides d_model / 32, so the steady-state loop
// issues its loads unconditionally and the compiler can count the outstanding loads exactly.
template <int KPRE, int OB>
__global__ __launch_bounds__(kMaxWaves * 64) void cache_write_packed_kernel(const WriteArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[kTokTile * kMaxWriteDModel];
  __shared__ float ssq_part[kMaxWaves][kTokTile];
  __shared__ int64_t tok_slot[kTokTile];
  // (cos, sin) of each token's pair angles; rows padded by one entry, so that the lanes of one
  // pair (one token each) hit different banks
  __shared__ f32x2 rope_cs[kTokTile][kMaxRopePairs + 1];

  const int nwave = blockDim.x >> 6;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, q = lane >> 4;
  const int dm = a.d_model, DC = a.d_c, DR = a.d_rope, NO = DC + DR;
  const int n_tok = a.geo.chunk_tokens;
  const int64_t M = (int64_t)a.batch * n_tok;    // tokens of the flat [batch][chunk] order
  const int64_t g0 = (int64_t)blockIdx.x * a.tok_per_wg;
  const int ntok = (int)(M - g0 < a.tok_per_wg ? M - g0 : a.tok_per_wg);  // >= 1 by the grid
  const int rows_pad = (ntok + 7) & ~7;
  const int ngrp = rows_pad / 8;                 // direct loads per column block
  VMLA_STAMP(a, kStampWritePacked, 0);

  // RMSNorm gain of this lane's outputs 32 wave + 16 ob + 4q .. +3, fetched first
  constexpr int OPW = 16 * OB;  // outputs per wave
  u32x2 gam[OB];
#pragma unroll
  for (int ob = 0; ob < OB; ++ob) {
    const int o = OPW * wave + 16 * ob + 4 * q;
    gam[ob] = u32x2{kOneBf16x2, kOneBf16x2};
    if (a.gamma && o + 4 <= DC) gam[ob] = *reinterpret_cast<const u32x2*>(a.gamma + o);
  }

  // ---- contraction order: k-step i of this workgroup is column k-step (i + rot) mod nks, rot
  // a whole column block, so that the workgroups of one L2 start at different weight lines ----
  const int nks = dm / 32, nblk = dm / 64;
  const int rotb = (int)((blockIdx.x >> 3) % (unsigned)nblk);
  const int rot = 2 * rotb;
  auto kstep = [&](int i) { const int k = i + rot; return k < nks ? k : k - nks; };
  // x arrives in two phases: k-steps [0, i_ph1) first, the rest during the first phase's work
  const int i_ph1 = (nks / 2) / KPRE * KPRE;     // 0: a single phase
  const int i_dma1 = i_ph1 > KPRE ? i_ph1 - KPRE : 0;

  // direct loads of the column blocks ib_begin .. ib_end-1 (in contraction order), rows past
  // the block's tokens repeating its last token (their results are never stored)
  auto issue_x = [&](int ib_begin, int ib_end) {
    const int n = (ib_end - ib_begin) * ngrp;
    for (int j = wave; j < n; j += nwave) {
      const int jb = j / ngrp, rg = j - jb * ngrp;
      int b = rotb + ib_begin + jb;
      if (b >= nblk) b -= nblk;
      const int t = rg * 8 + (lane >> 3), cs = lane & 7;
      const int cc = cs ^ ((t >> 1) & 7);
      const int tt = t < ntok ? t : ntok - 1;
      lds_dma16(a.x + (size_t)(g0 + tt) * dm + b * 64 + cc * 8,
                __builtin_amdgcn_readfirstlane(lds_addr(xs + (b * rows_pad + rg * 8) * 64)));
    }
  };
  issue_x(0, i_ph1 > 0 ? i_ph1 / 2 : nblk);

  // ---- this wave's packed panel: k-step k holds its two A operands (outputs 32 wave + 16 ob
  // + r, columns 32k + 8q ..) as 2 KB contiguous, lane-ordered ------------------------------
  const uint16_t* wpan = a.w_packed + ((size_t)wave * nks * OB) * 512 + lane * 8;
  u32x4 wb[KPRE][OB];
#pragma unroll
  for (int j = 0; j < KPRE; ++j) {
    const int k = kstep(j);
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) wb[j][ob] = ldg16(wpan + (OB * k + ob) * 512);
  }
  // while the first loads are in flight: each token's ring row (and slot), and the RoPE angles
  // with the pair index uniform across a wave, so that the angle table is read by scalar loads
  // (a per-lane index would turn them into vector loads that wait for every load in flight)
  const int npair = DR / 2;
  if (lane < ntok) {
    const int g = (int)g0 + lane;  // batch * chunk_tokens < 2^31 (validated on the host)
    const int b = g / n_tok, n = g - b * n_tok;
    const TokenPos pos = token_pos(a.geo, n);
    if (wave == 0) {
      const int64_t slot = ring_slot(a.geo, pos);
      tok_slot[lane] = (int64_t)b * a.geo.ring_tokens + slot;
      if (b == 0 && a.slots) a.slots[n] = (int32_t)slot;
    }
    for (int pr = wave; pr < npair; pr += nwave)  // identity with a sink
      rope_cs[lane][pr] = a.geo.sink_frames == 0 ? rope_cos_sin(a.rope, pr, pos) : f32x2{1.f, 0.f};
  }
  // loads complete in issue order: once at most the OB KPRE weight loads issued after them are
  // outstanding, this wave's first-phase x loads (and the gain) have landed
  wait_vmcnt<OB * KPRE>();
  __syncthreads();
  VMLA_STAMP(a, kStampWritePacked, 1);

  f32x4 acc[OB][2];  // [output block][token block]
#pragma unroll
  for (int ob = 0; ob < OB; ++ob)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) acc[ob][tb] = f32x4{};

  const int tmax = rows_pad - 1;
  auto mma_step = [&](int i, const u32x4 (&w)[OB]) {
    const int k = kstep(i);
    const int b = k >> 1, cc = 4 * (k & 1) + q;
    bf16x8 xb[2];
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const int t = 16 * tb + r < tmax ? 16 * tb + r : tmax;
      xb[tb] = as_bf16x8(*reinterpret_cast<const u32x4*>(&xs[xpos(b, t, cc, rows_pad) * 8]));
    }
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) acc[ob][tb] = mfma16(as_bf16x8(w[ob]), xb[tb], acc[ob][tb]);
  };
  auto steady = [&](int i0) {  // k-steps i0 .. i0+KPRE-1, refilling the ring KPRE ahead
#pragma unroll
    for (int j = 0; j < KPRE; ++j) {
      mma_step(i0 + j, wb[j]);
      const int kn = kstep(i0 + j + KPRE);
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) wb[j][ob] = ldg16(wpan + (OB * kn + ob) * 512);
    }
  };
  // the second phase's loads are issued KPRE k-steps before its first use, after the weight
  // loads of the k-steps that precede it (so that those do not wait for them); at k-step
  // i_ph1 the OB KPRE weight loads issued since are the only ones that may still be pending
  int i0 = 0;
  for (; i0 < i_dma1; i0 += KPRE) steady(i0);
  if (i_ph1 > 0) {
    issue_x(i_ph1 / 2, nblk);
    for (; i0 < i_ph1; i0 += KPRE) steady(i0);
    wait_vmcnt<OB * KPRE>();
    __syncthreads();
    VMLA_STAMP(a, kStampWritePacked, 2);
  }
  for (; i0 < nks - KPRE; i0 += KPRE) steady(i0);
#pragma unroll
  for (int j = 0; j < KPRE; ++j) mma_step(i0 + j, wb[j]);
  VMLA_STAMP(a, kStampWritePacked, 3);

  // ---- epilogue. Lane (r, q) holds, for token 16 tb + r of the block, outputs
  // OPW wave + 16 ob + 4q + e (e = 0..3) in acc[ob][tb][e] ---------------------------------
  float ss[2] = {0.f, 0.f};
#pragma unroll
  for (int ob = 0; ob < OB; ++ob)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int o = OPW * wave + 16 * ob + 4 * q + e;
        if (o < DC) ss[tb] += acc[ob][tb][e] * acc[ob][tb][e];
      }
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    ss[tb] += __shfl_xor(ss[tb], 16);
    ss[tb] += __shfl_xor(ss[tb], 32);
    if (q == 0) ssq_part[wave][16 * tb + r] = ss[tb];
  }
  __syncthreads();  // every wave is past its last x read: the tile area is reused below
  VMLA_STAMP(a, kStampWritePacked, 4);

  // normalized latents and rotated keys, rounded to bf16, into the tile ot[t][0 .. NO)
  const int ots = NO + 8;  // row stride (elements): 16 bytes of padding per row
  uint16_t* ot = xs;
  float tot[2], rstd[2];
  sum_wave_parts<kMaxWaves>(&ssq_part[0][0], kTokTile, nwave, r, tot);
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) rstd[tb] = a.gamma ? rsqrtf(tot[tb] / (float)DC + a.eps) : 1.f;
  write_out_tile(acc, gam, rstd, &rope_cs[0][0], kMaxRopePairs + 1, OPW * wave, DC, NO, r, q, ntok,
                 ot, ots);
  __syncthreads();
  VMLA_STAMP(a, kStampWritePacked, 5);

  // ---- stores: token t's row of NO/8 chunks (c_kv, then k_r) to its ring slot, coalesced ---
  const int cpt = NO / 8;
  for (int i = threadIdx.x; i < ntok * cpt; i += nwave * 64) {
    const int t = i / cpt, ch = i - t * cpt;
    const int64_t row = tok_slot[t];
    const u32x4 val = *reinterpret_cast<const u32x4*>(&ot[t * ots + ch * 8]);
    const int o = ch * 8;
    if (o < DC) stg16(a.c_kv + (size_t)row * DC + o, val);
    else stg16(a.k_r + (size_t)row * DR + (o - DC), val);
  }
  VMLA_STAMP_DRAINED(a, kStampWritePacked, 6);
}

// cache_write_wide_kernel (packed weights, more than 32 tokens per compute unit: batched calls).
// One workgroup per compute unit takes up to 16 TB tokens and all outputs, so that the weight
// panel, which every token needs whole, is streamed once per compute unit rather than once per
// 32 tokens. x no longer fits in LDS whole: it passes through a ring of three buffers of one
// phase each (KPRE / 2 k-steps of columns, in contraction order), filled by a loader wave (the
// last wave) that issues only these loads, so that it counts them exactly (a phase is a
// compile-time number of loads) while the compute waves' weight loads stay in flight. Two
// phases are in flight while a third is contracted, and one barrier per phase hands a buffer
// from the compute waves to the loader and back. The compute waves are those of
// cache_write_packed_kernel (one per 32 outputs, the same packed panel, the same MFMA), each with
// TB token blocks of accumulators. All waves share the tokens' ring rows and RoPE angles while
// the first phase lands, and every wave takes part in the stores. LDS (dynamic,
// cache_write_wide_lds_bytes): three x buffers [KPRE / 4 column blocks][16 TB rows][64],
// swizzled like the packed kernel's x tile (the output tile reuses them), then the per-wave sums
// of squares [waves - 1][16 TB], the ring rows [16 TB] and (cos, sin) [16 TB][d_rope / 2 + 1].
constexpr int kWideBufs = 3;

template <int KPRE, int TB>
__global__ __launch_bounds__(512) void cache_write_wide_kernel(const WriteArgs a) {
  constexpr int OB = 2, OPW = 16 * OB;
  constexpr int ROWS = 16 * TB;            // token rows of the x buffers (>= the block's tokens)
  constexpr int PK = KPRE / 2;             // k-steps per phase
  constexpr int PB = PK / 2;               // column blocks of 64 per phase
  constexpr int XB = PB * ROWS * 64;       // elements per x buffer
  constexpr int LPP = PB * ROWS / 8;       // loads per phase (1 KB each, all from the loader)
  static_assert(PK % 2 == 0 && 2 * LPP < 64, "two phases of loads within the vmcnt range");
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  const int nwave = blockDim.x >> 6, ncw = nwave - 1;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool loader = wave == ncw;
  const int r = lane & 15, q = lane >> 4;
  const int dm = a.d_model, DC = a.d_c, DR = a.d_rope, NO = DC + DR;
  const int n_tok = a.geo.chunk_tokens;
  const int64_t M = (int64_t)a.batch * n_tok;
  const int64_t g0 = (int64_t)blockIdx.x * a.tok_per_wg;
  const int ntok = (int)(M - g0 < a.tok_per_wg ? M - g0 : a.tok_per_wg);  // 1 .. ROWS
  const int nks = dm / 32, nblk = dm / 64;
  const int nph = nks / PK;                // phases (KPRE divides nks)
  const int npair = DR / 2;
  const int cs_ld = npair + 1;  // (cos, sin) row stride, padded as in the packed kernel
  uint16_t* xbuf = smem;
  float* ssq_part = reinterpret_cast<float*>(smem + kWideBufs * XB);
  int64_t* tok_slot = reinterpret_cast<int64_t*>(ssq_part + ncw * ROWS);
  f32x2* rope_cs = reinterpret_cast<f32x2*>(tok_slot + ROWS);

  // contraction order: k-step i is column k-step (i + rot) mod nks, rot a whole column block
  const int rotb = (int)((blockIdx.x >> 3) % (unsigned)nblk);
  const int rot = 2 * rotb;
  auto kstep = [&](int i) { const int k = i + rot; return k < nks ? k : k - nks; };
  VMLA_STAMP(a, kStampWriteWide, 0);

  // each token's ring row (and slot) and the (cos, sin) of its RoPE pair angles, computed by all
  // waves while the first phase of x lands: wave w takes the pairs w, w + nwave, .. (a pair index
  // uniform across the wave, so that the angle table is read by scalar loads) and wave 0, a
  // compute wave, the ring rows
  auto tables = [&]() {
    constexpr int NT = (ROWS + 63) / 64;  // tokens per lane
    TokenPos pos[NT];
#pragma unroll
    for (int k = 0; k < NT; ++k) {
      const int t = lane + 64 * k;
      const int g = (int)g0 + (t < ntok ? t : ntok - 1);  // < 2^31 (validated on the host)
      const int b = g / n_tok, n = g - b * n_tok;
      pos[k] = token_pos(a.geo, n);
      if (wave == 0 && t < ntok) {
        const int64_t slot = ring_slot(a.geo, pos[k]);
        tok_slot[t] = (int64_t)b * a.geo.ring_tokens + slot;
        if (b == 0 && a.slots) a.slots[n] = (int32_t)slot;
      }
    }
    for (int p = wave; p < npair; p += nwave) {
      // the pair index made visibly uniform, so that its table entries are read once, by scalar
      // loads (as a per-lane index they become vector loads that each wait for every load)
      const int pr = __builtin_amdgcn_readfirstlane(p);
#pragma unroll
      for (int k = 0; k < NT; ++k) {
        const int t = lane + 64 * k;
        const f32x2 cs =  // identity with a sink
            a.geo.sink_frames == 0 ? rope_cos_sin(a.rope, pr, pos[k]) : f32x2{1.f, 0.f};
        if (t < ntok) rope_cs[t * cs_ld + pr] = cs;
      }
    }
  };

  if (loader) {
    // phase p's columns into buffer p mod 3; rows past the block's tokens repeat its last token
    auto issue_x = [&](int p) {
      uint16_t* buf = xbuf + (p % kWideBufs) * XB;
#pragma unroll
      for (int j = 0; j < PB; ++j) {
        int b = rotb + p * PB + j;
        if (b >= nblk) b -= nblk;
#pragma unroll
        for (int rg = 0; rg < ROWS / 8; ++rg) {
          const int t = rg * 8 + (lane >> 3), cs = lane & 7;
          const int cc = cs ^ ((t >> 1) & 7);
          const int tt = t < ntok ? t : ntok - 1;
          lds_dma16(a.x + (size_t)(g0 + tt) * dm + b * 64 + cc * 8,
                    __builtin_amdgcn_readfirstlane(lds_addr(buf + (j * ROWS + rg * 8) * 64)));
        }
      }
    };
    issue_x(0);
    if (nph > 1) issue_x(1);
    tables();  // after the phase loads: a memory operation in it only makes the waits stricter
    for (int p = 0; p < nph; ++p) {
      // phase p has landed once at most the next phase's loads are outstanding (vector memory
      // operations complete in issue order)
      if (p + 1 < nph) wait_vmcnt<LPP>();
      else wait_vmcnt<0>();
      __syncthreads();  // phase p visible; the compute waves are done with phase p - 1
      if (p + 2 < nph) issue_x(p + 2);  // into the buffer phase p - 1 left
    }
    __syncthreads();  // the compute waves' sums of squares are in LDS
    __syncthreads();  // the output tile is complete
  } else {
    // RMSNorm gain of this lane's outputs OPW wave + 16 ob + 4q .. +3
    u32x2 gam[OB];
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) {
      const int o = OPW * wave + 16 * ob + 4 * q;
      gam[ob] = u32x2{kOneBf16x2, kOneBf16x2};
      if (a.gamma && o + 4 <= DC) gam[ob] = *reinterpret_cast<const u32x2*>(a.gamma + o);
    }
    // the tables first: issuing a weight ring's loads can stall this wave until the compute
    // unit's memory pipeline, which the loader's x loads fill first, has room for them
    tables();
    VMLA_STAMP(a, kStampWriteWide, 1);
    // this wave's packed panel slice (as in cache_write_packed_kernel), KPRE k-steps ahead
    const uint16_t* wpan = a.w_packed + ((size_t)wave * nks * OB) * 512 + lane * 8;
    u32x4 wb[KPRE][OB];
#pragma unroll
    for (int j = 0; j < KPRE; ++j) {
      const int k = kstep(j);
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) wb[j][ob] = ldg16(wpan + (OB * k + ob) * 512);
    }
    f32x4 acc[OB][TB];
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) acc[ob][tb] = f32x4{};
    // k-step jj of the phase in buffer `buf`: column block jj / 2, chunks 4 (jj & 1) + q
    auto mma_step = [&](const uint16_t* buf, int jj, const u32x4 (&w)[OB]) {
      const int j = jj >> 1, cc = 4 * (jj & 1) + q;
      bf16x8 xb[TB];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const int t = 16 * tb + r;
        xb[tb] = as_bf16x8(*reinterpret_cast<const u32x4*>(&buf[xpos(j, t, cc, ROWS) * 8]));
      }
#pragma unroll
      for (int ob = 0; ob < OB; ++ob)
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) acc[ob][tb] = mfma16(as_bf16x8(w[ob]), xb[tb], acc[ob][tb]);
    };
    // one pass = two phases = the KPRE k-steps of the weight ring. The refill is a compile-time
    // choice, so that the steady-state passes issue their loads on every path and the compiler
    // counts the outstanding loads exactly; a run-time condition would make it wait for all of
    // them (the whole ring) at every pass.
    auto pass = [&](int i0, auto refill) {
#pragma unroll
      for (int j = 0; j < KPRE; ++j) {
        const int ph = (i0 + j) / PK;
        if (j % PK == 0) __syncthreads();  // phase ph is in its buffer
        if (j % PK == 0 && ph < 10) VMLA_STAMP(a, kStampWriteWide, 2 + ph);
        mma_step(xbuf + (ph % kWideBufs) * XB, j % PK, wb[j]);
        if constexpr (decltype(refill)::value) {
          const int kn = kstep(i0 + j + KPRE);
#pragma unroll
          for (int ob = 0; ob < OB; ++ob) wb[j][ob] = ldg16(wpan + (OB * kn + ob) * 512);
        }
      }
    };
    int i0 = 0;
    for (; i0 < nks - KPRE; i0 += KPRE) pass(i0, std::true_type{});
    pass(i0, std::false_type{});
    VMLA_STAMP(a, kStampWriteWide, 12);
    // sums of squares of the latent outputs per token
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      float ss = 0.f;
#pragma unroll
      for (int ob = 0; ob < OB; ++ob)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int o = OPW * wave + 16 * ob + 4 * q + e;
          if (o < DC) ss += acc[ob][tb][e] * acc[ob][tb][e];
        }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      if (q == 0) ssq_part[wave * ROWS + 16 * tb + r] = ss;
    }
    __syncthreads();  // every wave is past its last x read: the output tile reuses the buffers
    VMLA_STAMP(a, kStampWriteWide, 13);
    // normalized latents and rotated keys, rounded to bf16, into the tile ot[t][0 .. NO)
    const int ots = NO + 8;
    uint16_t* ot = xbuf;
    float tot[TB];
    sum_wave_parts<7>(ssq_part, ROWS, ncw, r, tot);  // at most 8 waves, one of them the loader
    float rstd[TB];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) rstd[tb] = a.gamma ? rsqrtf(tot[tb] / (float)DC + a.eps) : 1.f;
    write_out_tile(acc, gam, rstd, rope_cs, cs_ld, OPW * wave, DC, NO, r, q, ntok, ot, ots);
    __syncthreads();  // the output tile is complete
    VMLA_STAMP(a, kStampWriteWide, 14);
  }

  // stores: token t's row of NO/8 chunks (c_kv, then k_r) to its ring slot, coalesced
  const int ots = NO + 8;
  const uint16_t* ot = xbuf;
  const int cpt = NO / 8;
  for (int i = threadIdx.x; i < ntok * cpt; i += nwave * 64) {
    const int t = i / cpt, ch = i - t * cpt;
    const int64_t row = tok_slot[t];
    const u32x4 val = *reinterpret_cast<const u32x4*>(&ot[t * ots + ch * 8]);
    const int o = ch * 8;
    if (o < DC) stg16(a.c_kv + (size_t)row * DC + o, val);
    else stg16(a.k_r + (size_t)row * DR + (o - DC), val);
  }
  VMLA_STAMP_DRAINED(a, kStampWriteWide, 15);
}

// Packed weight panel for cache_write_packed_kernel: W' = [W_DKV; W_KR; zero rows up to a whole
// number of wave slices of 16 OB rows]. Entry ((w * nks + k) * OB + ob) * 512 + 8 l + j holds
// W'[16 OB w + 16 ob + l % 16][32 k + 8 (l / 16) + j]: the MFMA 16x16x32 A operand of lane l for
// wave slice w, 16-row block ob and k-step k, so that every load of the kernel reads 1 KB
// contiguous. One thread per 16-byte entry.
__global__ __launch_bounds__(256) void pack_write_weights_kernel(const WriteArgs a) {
  const int dm = a.d_model, DC = a.d_c, NO = a.d_c + a.d_rope;
  const int nks = dm / 32;
  const int OB = write_blocks_per_wave(NO), OPW = 16 * OB;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;  // 16-byte entry
  const int64_t n_entries = (int64_t)((NO + OPW - 1) / OPW) * nks * OB * 64;
  if (e >= n_entries) return;
  const int l = (int)(e & 63);
  const int64_t blk = e >> 6;  // (w * nks + k) * OB + ob
  const int ob = (int)(blk % OB);
  const int64_t wk = blk / OB;
  const int k = (int)(wk % nks), w = (int)(wk / nks);
  const int o = OPW * w + 16 * ob + (l & 15);
  const int col = 32 * k + 8 * (l >> 4);
  u32x4 v = {0u, 0u, 0u, 0u};
  if (o < DC) v = ldg16(a.w_dkv + (size_t)o * dm + col);
  else if (o < NO) v = ldg16(a.w_kr + (size_t)(o - DC) * dm + col);
  stg16(a.w_packed_out + e * 8, v);
}

constexpr int kTok = 32;     // tokens per workgroup
constexpr int kWaves = 4;
constexpr int kKC = 64;      // contraction columns per stage: 8 chunks of 16 B per row

// Position (16 B units) of chunk c of staged row r: row-major with 8 chunks per row, the chunk
// index XOR-ed with (r / 2) mod 8, so 16 consecutive rows read at one chunk hit distinct banks.
__device__ __forceinline__ int swz(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

template <int NB>  // 32-wide output blocks covering d_c + d_rope
__global__ __launch_bounds__(kWaves * 64) void cache_write_staged_kernel(const WriteArgs a) {
  constexpr int ROWS = NB * 32 + kTok;        // staged rows: weight rows, then x rows
  constexpr int INSTR = ROWS * 8 / 64;        // 1 KB load instructions per stage
  constexpr int PER_WAVE = (INSTR + kWaves - 1) / kWaves;
  constexpr int MAXB = (NB + kWaves - 1) / kWaves;  // output blocks per wave
  // LDS stages (kStages - 1 chunks in flight): four while they fit in 150 KB, else three
  constexpr int kStages = ROWS * kKC * 2 * 4 <= 150 * 1024 ? 4 : 3;
  static_assert(ROWS % 8 == 0, "stage is a whole number of 1 KB loads");
  static_assert(INSTR % kWaves == 0, "every wave issues the same number of loads per stage");
  __shared__ __attribute__((aligned(16))) uint16_t stage[kStages][ROWS * kKC];
  __shared__ float ssq_part[kWaves][kTok];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches, SGPR m0
  const int g = lane >> 5, l32 = lane & 31;
  const int b = blockIdx.y;
  const int n0 = blockIdx.x * kTok;
  const int dm = a.d_model, DC = a.d_c, DR = a.d_rope;
  const int n_tok = a.geo.chunk_tokens;

  // Global source of each of this wave's load instructions (instruction j = wave + kWaves*i):
  // its lane covers LDS position p = j*64 + lane = (row r, swizzled chunk); rows past the
  // weights or the chunk read a valid row whose results are discarded.
  const uint16_t* src[PER_WAVE];
#pragma unroll
  for (int i = 0; i < PER_WAVE; ++i) {
    const int j = wave + kWaves * i;
    const int p = (j < INSTR ? j : 0) * 64 + lane;
    const int r = p >> 3, cs = p & 7;
    const int c = cs ^ ((r >> 1) & 7);  // logical chunk stored at this position
    const uint16_t* row;
    if (r < NB * 32) {
      row = r < DC ? a.w_dkv + (size_t)r * dm
                   : (r < DC + DR ? a.w_kr + (size_t)(r - DC) * dm : a.w_dkv);
    } else {
      const int n = n0 + (r - NB * 32);
      row = a.x + ((size_t)b * n_tok + (n < n_tok ? n : 0)) * dm;
    }
    src[i] = row + c * 8;
  }
  auto issue = [&](int chunk) {
    uint16_t* st = stage[chunk % kStages];
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int j = wave + kWaves * i;
      if (INSTR % kWaves == 0 || j < INSTR)
        lds_dma16(src[i] + chunk * kKC, __builtin_amdgcn_readfirstlane(lds_addr(st + j * 512)));
    }
  };

  f32x16 acc[MAXB];
#pragma unroll
  for (int m = 0; m < MAXB; ++m) acc[m] = f32x16{};

  const int nchunks = dm / kKC;
#pragma unroll
  for (int c = 0; c < kStages - 1; ++c)
    if (c < nchunks) issue(c);
  for (int i = 0; i < nchunks; ++i) {
    // chunk i has landed once at most (kStages - 2) later chunks are still outstanding
    if (i + kStages - 2 < nchunks) wait_vmcnt<(kStages - 2) * PER_WAVE>();
    else wait_vmcnt<0>();
    __syncthreads();  // all waves' parts of chunk i are in LDS; chunk i-1 is no longer read
    if (i + kStages - 1 < nchunks) issue(i + kStages - 1);
    const uint16_t* st = stage[i % kStages];
#pragma unroll
    for (int ks = 0; ks < kKC / 16; ++ks) {
      const int c = ks * 2 + g;
      const bf16x8 bx = as_bf16x8(*reinterpret_cast<const u32x4*>(&st[swz(NB * 32 + l32, c) * 8]));
#pragma unroll
      for (int m = 0; m < MAXB; ++m) {
        // a wave with fewer blocks repeats the last one (discarded) instead of branching
        const int ob = wave + kWaves * m < NB ? wave + kWaves * m : NB - 1;
        const bf16x8 aw =
            as_bf16x8(*reinterpret_cast<const u32x4*>(&st[swz(ob * 32 + l32, c) * 8]));
        acc[m] = mfma32(aw, bx, acc[m]);
      }
    }
  }

  // ---- epilogue: lane holds token l32, outputs ob*32 + 8i + 4g + j of its blocks ----------
  float ss = 0.f;
#pragma unroll
  for (int m = 0; m < MAXB; ++m) {
    const int ob = wave + kWaves * m;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int o = ob * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
      if (ob < NB && o < DC) ss += acc[m][r] * acc[m][r];
    }
  }
  ss = half_swap_sum(ss);
  if (g == 0) ssq_part[wave][l32] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) tot += ssq_part[w][l32];
  const float rstd = a.gamma ? rsqrtf(tot / (float)DC + a.eps) : 1.f;

  const int n = n0 + l32;
  if (n >= n_tok) return;
  const TokenPos pos = token_pos(a.geo, n);
  const int64_t slot = ring_slot(a.geo, pos);
  uint16_t* cdst = a.c_kv + ((size_t)b * a.geo.ring_tokens + slot) * DC;
  uint16_t* kdst = a.k_r + ((size_t)b * a.geo.ring_tokens + slot) * DR;
#pragma unroll
  for (int m = 0; m < MAXB; ++m) {
    const int ob = wave + kWaves * m;
    if (ob >= NB) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = ob * 32 + 8 * i + 4 * g;  // first of 4 consecutive outputs
      float v[4] = {acc[m][4 * i], acc[m][4 * i + 1], acc[m][4 * i + 2], acc[m][4 * i + 3]};
      if (o + 4 <= DC) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] *= rstd;
          if (a.gamma) v[e] *= bf16_bits_to_f32(a.gamma[o + e]);
        }
        const f32x4 fv = {v[0], v[1], v[2], v[3]};
        *reinterpret_cast<bf16x4*>(cdst + o) = to_bf16x4(fv);
      } else if (o >= DC && o + 4 <= DC + DR) {
        const int ch = o - DC;  // channels ch .. ch+3 = RoPE pairs ch/2 and ch/2 + 1
        if (a.geo.sink_frames == 0) {  // with a sink the ring keeps the unrotated key
          const f32x2 c0 = rope_cos_sin(a.rope, ch / 2, pos);
          const f32x2 c1 = rope_cos_sin(a.rope, ch / 2 + 1, pos);
          const float r0 = v[0] * c0[0] - v[1] * c0[1], r1 = v[0] * c0[1] + v[1] * c0[0];
          const float r2 = v[2] * c1[0] - v[3] * c1[1], r3 = v[2] * c1[1] + v[3] * c1[0];
          v[0] = r0, v[1] = r1, v[2] = r2, v[3] = r3;
        }
        const f32x4 fv = {v[0], v[1], v[2], v[3]};
        *reinterpret_cast<bf16x4*>(kdst + ch) = to_bf16x4(fv);
      }
    }
  }
  if (a.slots && b == 0 && wave == 0 && g == 0) a.slots[n] = (int32_t)slot;
}

}  // namespace

static hipError_t launch_cache_write_staged(const WriteArgs& a, hipStream_t s) {
  // validated by the caller: d_model % 64 == 0, d_c % 16 == 0, d_rope % 8 == 0,
  // d_c + d_rope <= 288
  const int nb = (a.d_c + a.d_rope + 31) / 32;
  const dim3 grid((a.geo.chunk_tokens + kTok - 1) / kTok, a.batch);
  const dim3 block(kWaves * 64);
  switch (nb) {
    case 1: hipLaunchKernelGGL(cache_write_staged_kernel<1>, grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL(cache_write_staged_kernel<2>, grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL(cache_write_staged_kernel<3>, grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL(cache_write_staged_kernel<4>, grid, block, 0, s, a); break;
    case 5: hipLaunchKernelGGL(cache_write_staged_kernel<5>, grid, block, 0, s, a); break;
    case 6: hipLaunchKernelGGL(cache_write_staged_kernel<6>, grid, block, 0, s, a); break;
    case 7: hipLaunchKernelGGL(cache_write_staged_kernel<7>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(cache_write_staged_kernel<8>, grid, block, 0, s, a); break;
    case 9: hipLaunchKernelGGL(cache_write_staged_kernel<9>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int cache_write_tokens_per_wg(int64_t tokens, int n_cu) {
  // one workgroup per CU while that keeps blocks within the 32-row tile, else full tiles
  const int64_t per = (tokens + n_cu - 1) / n_cu;
  return (int)(per < 1 ? 1 : (per > kTokTile ? kTokTile : per));
}

namespace {
constexpr int kWideMaxTokens = 80;  // 5 token blocks of 16 per workgroup

// The wide kernel's KPRE for these dims, or 0 when it does not apply: packed weights with 32
// outputs per wave and at most 7 compute waves (d_c + d_rope <= 224), d_model a multiple of
// 384 or 256, and more than 32 tokens per compute unit.
int wide_kpre(const WriteArgs& a, int n_cu) {
  const int no = a.d_c + a.d_rope, nks = a.d_model / 32;
  if (!a.w_packed || write_blocks_per_wave(no) != 2 || (no + 31) / 32 > 7) return 0;
  if ((int64_t)a.batch * a.geo.chunk_tokens <= (int64_t)kTokTile * n_cu) return 0;
  return nks % 12 == 0 ? 12 : nks % 8 == 0 ? 8 : 0;
}

size_t cache_write_wide_lds_bytes(int kpre, int tb, int ncw, int npair) {
  const size_t rows = 16 * (size_t)tb;
  return kWideBufs * (size_t)(kpre / 4) * rows * 64 * 2 + ncw * rows * 4 + rows * 8 +
         rows * (npair + 1) * 8;
}

template <int KPRE>
hipError_t launch_wide(const WriteArgs& a, int n_cu, hipStream_t s) {
  WriteArgs b = a;
  const int64_t M = (int64_t)a.batch * a.geo.chunk_tokens;
  const int64_t per = (M + n_cu - 1) / n_cu;
  b.tok_per_wg = (int)(per > kWideMaxTokens ? kWideMaxTokens : per);
  const int tb = (b.tok_per_wg + 15) / 16;
  const int ncw = (a.d_c + a.d_rope + 31) / 32;
  const size_t lds = cache_write_wide_lds_bytes(KPRE, tb, ncw, a.d_rope / 2);
  const dim3 grid((unsigned)((M + b.tok_per_wg - 1) / b.tok_per_wg)), block((ncw + 1) * 64);
  auto go = [&](auto kernel) {
    // dynamic LDS beyond the default limit (up to 136 KB at the Wan shape)
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kernel, grid, block, lds, s, b);
    return hipGetLastError();
  };
  switch (tb) {
    case 3: return go(cache_write_wide_kernel<KPRE, 3>);
    case 4: return go(cache_write_wide_kernel<KPRE, 4>);
    default: return go(cache_write_wide_kernel<KPRE, 5>);
  }
}
}  // namespace

size_t write_weights_packed_elems(int d_model, int d_c, int d_rope) {
  const int ob = write_blocks_per_wave(d_c + d_rope), opw = 16 * ob;
  return (size_t)((d_c + d_rope + opw - 1) / opw) * (d_model / 32) * ob * 512;
}

hipError_t launch_pack_write_weights(const WriteArgs& a, hipStream_t s) {
  const int64_t entries = (int64_t)write_weights_packed_elems(a.d_model, a.d_c, a.d_rope) / 8;
  hipLaunchKernelGGL(pack_write_weights_kernel, dim3((unsigned)((entries + 255) / 256)), dim3(256),
                     0, s, a);
  return hipGetLastError();
}

hipError_t launch_cache_write(const WriteArgs& a, hipStream_t s) {
  if (!a.w_packed) return launch_cache_write_staged(a, s);
  if (const int kpre = wide_kpre(a, a.n_cu)) {  // batched calls: the panel once per compute unit
    return kpre == 12 ? launch_wide<12>(a, a.n_cu, s) : launch_wide<8>(a, a.n_cu, s);
  }
  // validated by the caller: d_model % 64 == 0, d_model <= kMaxWriteDModel, d_c % 16 == 0,
  // d_rope % 8 == 0, d_c + d_rope <= 576, 1 <= tok_per_wg <= 32
  const int ob = write_blocks_per_wave(a.d_c + a.d_rope);
  const int nw = (a.d_c + a.d_rope + 16 * ob - 1) / (16 * ob);
  const int nks = a.d_model / 32;  // even
  const int64_t M = (int64_t)a.batch * a.geo.chunk_tokens;
  const dim3 grid((unsigned)((M + a.tok_per_wg - 1) / a.tok_per_wg)), block(nw * 64);
  if (nw > kMaxWaves) return hipErrorInvalidValue;
  if (ob == 2) {
    if (nks % 12 == 0)
      hipLaunchKernelGGL((cache_write_packed_kernel<12, 2>), grid, block, 0, s, a);
    else if (nks % 8 == 0)
      hipLaunchKernelGGL((cache_write_packed_kernel<8, 2>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((cache_write_packed_kernel<2, 2>), grid, block, 0, s, a);
  } else {  // 64 outputs per wave: fewer k-steps in flight keep the register count in bounds
    if (nks % 4 == 0)
      hipLaunchKernelGGL((cache_write_packed_kernel<4, 4>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((cache_write_packed_kernel<2, 4>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace vmla
