// Latent attention of one chunk over the ring (Section "Inference-Time Reparameterization").
//
//   q_absorb      q_cat[row] = [ W_UK_h^T q_nope | RoPE_3D(q_R) | 0 pad ] * scale * log2(e)
//                 (query absorption, Eq. 8 in per-head form; Eq. 6; Eq. 7's scale)
//   latent_attend S^T = [c_kv | k_r] q_cat^T, online softmax in base 2, O_lat^T += c_kv^T P^T,
//                 over one key range (split) of the valid ring slots; writes the unnormalized
//                 O_lat and the running (max, sum) of every row
//   out_proj      merges the splits exactly, divides by the sum and applies W_UV_h (Eq. 2 /
//                 Eq. 10 without W_O)
//
// Rows are (batch, chunk token, head) triples in that order: row = (b*Nq + n)*H + h, so the
// query, workspace and output tensors are all addressed by one row index. Every head of every
// token reads the same ring tile: the heads are folded into the query rows (the cache is
// head-shared), so each [c_kv | k_r] tile is staged in LDS once per workgroup and serves all
// its rows.
#include <type_traits>
#include "vmla_device.h"

namespace vmla {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

// ---------------------------------------------------------------------------------------------
// q_absorb: grid (ceil(Nq/128), H, B), 4 waves, 32 tokens per wave, one head per workgroup.
// out^T[c][token] = W_UK_h^T[c][k] q_nope^T[k][token]; W_UK_h ([d_nope][d_c] row-major) is
// staged in LDS and read transposed with ds_read_b64_tr_b16, each lane's q_nope row is loaded
// once (all d_nope <= kMaxNope dims) and feeds every 32-wide output block.
// ---------------------------------------------------------------------------------------------
constexpr int kMaxNope = 128;

template <int DC> struct AbsorbChunk {  // W_UK_h columns staged in LDS per pass
  static constexpr int DCP = (DC + 31) / 32 * 32;
  static constexpr int CW = DCP <= 192 ? DCP : 128;
  static_assert(DCP % CW == 0, "whole column chunks");
  // single pass: the output rows go through an LDS tile (per wave 32 rows of DQKP + 8) that
  // reuses the W_UK_h area, and are stored whole
  static constexpr bool STAGE = DCP == CW;
};

template <int DC, int DR>
__global__ __launch_bounds__(256) void q_absorb_kernel(const AttendArgs a) {
  constexpr int DCP = AbsorbChunk<DC>::DCP;
  constexpr int CW = AbsorbChunk<DC>::CW;  // columns per pass (LDS holds d_nope x CW)
  constexpr int WS = CW + 8;               // LDS row stride (elements)
  constexpr int DQKP = (DC + DR + 15) / 16 * 16;
  constexpr int NCB = CW / 32;
  constexpr int KN = kMaxNope / 16;
  extern __shared__ __attribute__((aligned(16))) uint16_t wuk[];  // [d_nope][WS]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, l32 = lane & 31;
  const int h = blockIdx.y, b = blockIdx.z;
  const int H = a.n_heads, dn = a.d_nope, Nq = a.geo.q_count;
  const int nks = dn / 16;

  const int n = blockIdx.x * 128 + wave * 32 + l32;
  const bool ok = n < Nq;
  VMLA_STAMP(a, kStampQAbsorb, 0);
  const size_t row = ((size_t)b * Nq + (ok ? n : 0)) * H + h;
  const uint16_t* qn = a.q_nope + row * dn;
  uint16_t* dst = a.qcat + row * DQKP;

  // this lane's query row, B-operand layout (dims ks*16 + 8g .. +8), issued before the W wait.
  // The loads are unconditional: a lane past the chunk reads token 0's row and stores nothing,
  // and the steps ks >= nks, which read the last step again, feed no MFMA.
  bf16x8 bq[KN];
#pragma unroll
  for (int ks = 0; ks < KN; ++ks) bq[ks] = as_bf16x8(ldg16(qn + min(ks, nks - 1) * 16 + 8 * g));
  // the RoPE part's (u, v) pairs of this lane (pair p = lane mod NP of tokens tok0 + lane / NP +
  // TPI j), loaded now so that their latency passes under the contraction; tokens past the
  // chunk read the last token and are not written
  constexpr int NP = DR / 2;
  constexpr bool PAIR_PER_LANE = 64 % NP == 0;
  constexpr int TPI = PAIR_PER_LANE ? 64 / NP : 1, NIT = (32 + TPI - 1) / TPI;
  const int tok0 = blockIdx.x * 128 + wave * 32;
  uint32_t qraw[PAIR_PER_LANE ? NIT : 1];
  RopePair rp{};
  if constexpr (PAIR_PER_LANE) {
    rp = rope_pair(a.rope, lane % NP);  // a per-lane read of the kernel arguments: issued early too
#pragma unroll
    for (int j = 0; j < NIT; ++j) {
      const int t = min(tok0 + lane / NP + TPI * j, Nq - 1);
      qraw[j] = *reinterpret_cast<const uint32_t*>(a.q_r + (((size_t)b * Nq + t) * H + h) * DR + 2 * (lane % NP));
    }
  }
  // the rotation positions (frame, row, column) of the wave's 32 tokens, computed once per token
  // by lanes 0..31 while the loads are in flight (the divisions that split a token index into
  // its position would otherwise be repeated by every lane that rotates one of its pairs)
  __shared__ double qpos[4][3][32];
  if (lane < 32) {
    const TokenPos tp = rope_pos(a.geo, query_pos(a.geo, min(tok0 + lane, Nq - 1)));
    qpos[wave][0][lane] = (double)tp.f;
    qpos[wave][1][lane] = (double)tp.y;
    qpos[wave][2][lane] = (double)tp.x;
  }

  const uint16_t* wsrc = a.w_uk + (size_t)h * dn * DC;
  constexpr bool STAGE = AbsorbChunk<DC>::STAGE;
  constexpr int OS = DQKP + 8;  // output tile row stride (elements)
  uint16_t* ot = wuk + wave * 32 * OS;
  // tr-read addressing inside a 16-lane group
  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  for (int c0 = 0; c0 < DCP; c0 += CW) {
    const int cw = DC - c0 < CW ? DC - c0 : CW;  // real columns of this pass
    if (c0 > 0) __syncthreads();                 // the previous pass's reads are done
    {  // every staging load of this thread issued, then stored
      constexpr int PER = kMaxNope * (CW / 8) / 256;
      u32x4 wv[PER];
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int c = tid + 256 * i;
        if (c < dn * (cw / 8)) wv[i] = ldg16(wsrc + (size_t)(c / (cw / 8)) * DC + c0 + (c % (cw / 8)) * 8);
      }
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int c = tid + 256 * i;
        if (c < dn * (cw / 8)) *reinterpret_cast<u32x4*>(&wuk[(c / (cw / 8)) * WS + (c % (cw / 8)) * 8]) = wv[i];
      }
    }
    __syncthreads();
    if (c0 == 0) VMLA_STAMP(a, kStampQAbsorb, 1);

    f32x16 acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[cb] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KN; ++ks) {
      if (ks < nks) {
        const int k0 = ks * 16 + 8 * g;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const i16x4 lo = lds_read_tr(&wuk[(k0 + tr_row) * WS + cb * 32 + tr_col]);
          const i16x4 hi = lds_read_tr(&wuk[(k0 + 4 + tr_row) * WS + cb * 32 + tr_col]);
          acc[cb] = mfma32(join_bf16x8(lo, hi), bq[ks], acc[cb]);
        }
      }
    }
    if (c0 == 0) VMLA_STAMP(a, kStampQAbsorb, 2);
    if (STAGE) __syncthreads();  // every wave is done reading W_UK_h: its area holds the rows
    if (ok || STAGE) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = c0 + cb * 32 + 8 * i + 4 * g;
          if (c < DC) {
            const f32x4 v = {acc[cb][4 * i] * a.qscale, acc[cb][4 * i + 1] * a.qscale,
                             acc[cb][4 * i + 2] * a.qscale, acc[cb][4 * i + 3] * a.qscale};
            *reinterpret_cast<bf16x4*>(STAGE ? ot + l32 * OS + c : dst + c) = to_bf16x4(v);
          }
        }
    }
  }

  VMLA_STAMP(a, kStampQAbsorb, 3);

  // RoPE part and zero padding: 32 tokens x (DR/2) pairs per wave.
  auto rope_one = [&](int t, int p, const RopePair& rp, uint32_t raw) {
    const size_t r = ((size_t)b * Nq + t) * H + h;
    float u = bf16_bits_to_f32((uint16_t)(raw & 0xffff)), v = bf16_bits_to_f32((uint16_t)(raw >> 16));
    rotate_by(rope_cos_sin_at(qpos[wave][rp.axis][t - tok0], rp.theta), u, v);
    const uint32_t packed =
        (uint32_t)to_bf16_bits(u * a.qscale) | ((uint32_t)to_bf16_bits(v * a.qscale) << 16);
    *reinterpret_cast<uint32_t*>(STAGE ? ot + (t - tok0) * OS + DC + 2 * p
                                       : a.qcat + r * DQKP + DC + 2 * p) = packed;
  };
  if constexpr (PAIR_PER_LANE) {
    // lane l keeps pair l mod NP for all its tokens, so that it reads that pair's table entries
    // once (a per-iteration read would be a vector load waiting for every load in flight)
    const int p = lane % NP;
#pragma unroll
    for (int j = 0; j < NIT; ++j) {
      const int t = tok0 + lane / NP + TPI * j;
      if (t < tok0 + 32 && t < Nq) rope_one(t, p, rp, qraw[j]);
    }
  } else {
    for (int it = lane; it < 32 * NP; it += 64) {
      const int t = tok0 + it / NP, p = it % NP;
      if (t < Nq)
        rope_one(t, p, rope_pair(a.rope, p),
                 *reinterpret_cast<const uint32_t*>(a.q_r + (((size_t)b * Nq + t) * H + h) * DR + 2 * p));
    }
  }
  if (DQKP > DC + DR) {
    for (int t = tok0 + lane; t < tok0 + 32 && t < Nq; t += 64) {
      const size_t r = ((size_t)b * Nq + t) * H + h;
      for (int c = DC + DR; c < DQKP; ++c) {
        if (STAGE) ot[(t - tok0) * OS + c] = 0;
        else a.qcat[r * DQKP + c] = 0;
      }
    }
  }
  VMLA_STAMP(a, kStampQAbsorb, 4);
  if constexpr (STAGE) {
    __syncthreads();  // the wave's rows are complete in its tile
    VMLA_STAMP(a, kStampQAbsorb, 5);
    constexpr int CPR = DQKP / 8;  // 16-byte chunks per row
    for (int i = lane; i < 32 * CPR; i += 64) {
      const int t = i / CPR, k = i - t * CPR;
      if (tok0 + t < Nq)
        *reinterpret_cast<u32x4*>(a.qcat + (((size_t)b * Nq + tok0 + t) * H + h) * DQKP + k * 8) =
            *reinterpret_cast<const u32x4*>(&ot[t * OS + k * 8]);
    }
  }
  VMLA_STAMP_DRAINED(a, kStampQAbsorb, 6);
}

// ---------------------------------------------------------------------------------------------
// rope_window (attention sink only): the ring holds unrotated positional keys; rotate the keys
// of every valid slot at their window-local time (App. "Long-Horizon RoPE Re-indexing") into
// k_rot, which the attention kernel then reads in place of the ring. One thread per (slot,
// RoPE pair). Slot s holds frame slot fs = s / HW: a sink frame (fs < S, local time fs) or the
// recent frame f with S + (f - S) mod L = fs (L = W - S), whose local time is
// S + (f - local_lo) = S + ((fs - S) - (local_lo - S)) mod L.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void rope_window_kernel(const AttendArgs a) {
  const int np = a.d_rope / 2;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int b = blockIdx.y;
  if (e >= (int64_t)a.n_valid * np) return;
  const int64_t slot = e / np;
  const int p = (int)(e % np);
  const Geometry& g = a.geo;
  const int hw = g.grid_h * g.grid_w;
  const int fs = (int)(slot / hw), r = (int)(slot % hw);
  const int S = g.sink_frames, L = g.window_frames - S;
  TokenPos pos;
  if (fs < S) {
    pos.f = fs;
  } else {
    const int64_t d = ((int64_t)(fs - S) - (g.local_lo - S)) % L;
    pos.f = S + (d < 0 ? d + L : d);
  }
  pos.y = r / g.grid_w;
  pos.x = r % g.grid_w;
  const size_t off = ((size_t)b * g.ring_tokens + slot) * a.d_rope + 2 * p;
  const uint32_t raw = *reinterpret_cast<const uint32_t*>(a.k_r + off);
  float u = bf16_bits_to_f32((uint16_t)(raw & 0xffff)), v = bf16_bits_to_f32((uint16_t)(raw >> 16));
  rope_rotate(a.rope, p, pos, u, v);
  *reinterpret_cast<uint32_t*>(a.k_rot + off) =
      (uint32_t)to_bf16_bits(u) | ((uint32_t)to_bf16_bits(v) << 16);
}

// ---------------------------------------------------------------------------------------------
// bal_prep (adaptive partition only): one wave, launched before the attention kernel of an
// adaptive call. It reads the weights and per-workgroup durations the previous adaptive call on
// this workspace left, and sets each XCD's weight proportional to the units per time its
// workgroups achieved there (weight over the XCD's slowest workgroup time), normalized to a
// mean of kBalOne and clamped to [kBalMin, kBalMax]; equal weights when the record is missing,
// was made for another G, or lacks a duration. It then writes G and the marker, and clears the
// durations, which the attention kernel of this call fills in. Lane l reads and clears the
// durations of workgroups k = l mod 64 (XCD k mod 8 = l mod 8), so every duration is read and
// cleared by the same lane.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(64) void bal_prep_kernel(uint32_t* st, int G) {
  const int lane = threadIdx.x;
  uint32_t w_prev[8];
  bal_weights(st, G, w_prev);
  const bool hdr = st[9] == kBalMark && st[8] == (uint32_t)G;
  uint32_t tmax = 0, tmin = 0xffffffffu;
  for (int k = lane; k < G; k += 64) {
    const uint32_t t = st[kBalHead + k];
    tmax = max(tmax, t);
    tmin = min(tmin, t);
  }
  // combine the lanes of one XCD (lanes x, x + 8, .., x + 56)
#pragma unroll
  for (int sh = 8; sh < 64; sh <<= 1) {
    tmax = max(tmax, (uint32_t)__shfl_xor((int)tmax, sh));
    tmin = min(tmin, (uint32_t)__shfl_xor((int)tmin, sh));
  }
  // every lane gathers the 8 per-XCD results (XCD x from lane x)
  bool ok = hdr;
  double sp[8], tot = 0.0;
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const uint32_t mx = (uint32_t)__shfl((int)tmax, x), mn = (uint32_t)__shfl((int)tmin, x);
    const int nx = G > x ? (G - x + 7) / 8 : 0;  // workgroups on XCD x
    sp[x] = 0.0;
    if (nx > 0) {
      ok = ok && mn > 0u && mx < 1000000000u;
      sp[x] = (double)w_prev[x] / (double)(mx > 0u ? mx : 1u);
      tot += nx * sp[x];
    }
  }
  uint32_t w_new[8];
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const double v = ok && sp[x] > 0.0 ? kBalOne * sp[x] * G / tot : (double)kBalOne;
    w_new[x] = (uint32_t)fmin(fmax(rint(v), (double)kBalMin), (double)kBalMax);
  }
  for (int k = lane; k < G; k += 64) st[kBalHead + k] = 0u;
  if (lane < 10) st[lane] = lane < 8 ? w_new[lane] : lane == 8 ? (uint32_t)G : kBalMark;
}

// ---------------------------------------------------------------------------------------------
// latent_attend: grid G (about one workgroup per CU), NW waves, QB 32-row query blocks per wave.
//   LDS: a ring of three BN-token tiles [c_kv | k_r | pad], token-major. Iteration t computes
//   the scores of tile t+1 while the softmax of tile t runs on the VALU, then accumulates
//   PV of tile t, and stages tile t+2 from registers loaded at the top of the iteration.
//   S^T (keys x queries) = MFMA(A = K tile rows from LDS, B = q_cat rows in registers); each
//   lane then holds one query's scores for 16 keys per 32-key block, so the row max and sum
//   need only one exchange with lane l^32. P^T feeds the PV MFMA directly as the B operand,
//   and V^T (the c_kv columns of the same tile) is read with LDS transpose reads. Both the K
//   and the V operand of each MFMA are shared by the QB query blocks of the wave.
//   The running max is raised only when a tile's max exceeds it by more than kLazyMax (in
//   log2 units), so probabilities stay below 2^kLazyMax and the accumulators are rescaled
//   rarely; the final merge divides by the matching sum, so the result is unchanged.
//   Tiles go from global memory straight into LDS (global_load_lds, no registers), two tiles
//   ahead of their PV step. The (batch, row block, key tile) units are split evenly over the
//   workgroups (a row block may be shared by two or three of them), so every CU gets the same
//   amount of work.
// ---------------------------------------------------------------------------------------------
constexpr float kLazyMax = 8.0f;


// Tile layouts. Latent (DENSE = false): a tile row is [c_kv (DC) | k_r (DR) | pad], the scores
// contract over all of it and V is its first DC columns. Per-head rows (DENSE = true, DC = key
// width, DR = 0, DVW = value width, 0 meaning DC): a tile row is [K_h | V_h] of one head, the
// scores contract over K_h and V is the rest (the dense comparator: 128 | 128; the materialized
// form: [W_UK,h c ; k^R] | W_UV,h c = 128 | 128 or 160 | 128).
//
// Pair split (VS = 2, latent rows only): the waves of a pair share their 32 query rows. Each
// contracts the scores over its half of the [c_kv | k_r] columns, the two partial score tiles
// are exchanged through LDS at the step's barrier and summed (in the same order of operands on
// both sides, so both hold bitwise identical scores, running max and sum), and each wave
// accumulates the PV product for its half of the value columns. This halves the accumulator and
// query registers per wave, for latent widths whose 32 x d_c fp32 accumulators would not fit
// one wave, without computing any score twice.
template <int DC, int DR, int QB, int NW, int BN, bool DENSE = false, int DVW = 0, int VS = 1>
struct AttCfg {
  static constexpr int DQK = DC + DR;
  static constexpr int DQKP = (DQK + 15) / 16 * 16;
  static constexpr int KSTEPS = DQKP / 16;
  static constexpr int NSH = KSTEPS / VS;  // score steps of one wave
  static constexpr int OW = DENSE && DVW ? DVW : DC;  // value (and partial-result) width
  static constexpr int DVB = (OW + 31) / 32;
  static constexpr int DVBW = DVB / VS;               // value blocks per wave
  static constexpr int KB = BN / 32;       // 32-key blocks per tile
  static constexpr int VOFF = DENSE ? DQKP : 0;  // first V column of a tile row
  // Tile rows have no padding. Rows whose chunk count is a multiple of 16 bank groups (the
  // dense 128 | 128 rows, 32 chunks): chunk index XOR (4 (r mod 4) + (r / 4) mod 4) within
  // groups of 16. Other rows (latent DQKP elements; 160 | 128 = 36 chunks): chunk index XOR
  // ((r / 4) mod 4) within groups of 4. Either way the 16-row operand reads of the score MFMA
  // and the 4-row transpose reads of the PV MFMA hit 16 distinct 4-bank groups each (checked by
  // enumeration on the host for every layout instantiated here).
  static constexpr int STRIDE = DENSE ? DQKP + OW : DQKP;
  static constexpr int NT = NW * 64;
  static constexpr int ROWS = NW / VS * QB * 32;
  static_assert(VS == 1 || (VS == 2 && !DENSE && DVB % VS == 0 && NW % VS == 0 &&
                            KSTEPS % VS == 0 && QB == 1 && BN == 32), "pair split");
  static constexpr int OCT_C = DC / 8, OCT_R = DR / 8;
  static constexpr int CPR = STRIDE / 8;          // 16-byte chunks per tile row
  static constexpr int NDMA = BN * CPR / 64;      // 1 KB direct-to-LDS loads per tile
  static constexpr int DMA_PER_WAVE = (NDMA + NW - 1) / NW;
  static constexpr int TILE = BN * STRIDE;
  static constexpr int NBUF = 3;
  static_assert(DC % 8 == 0 && DR % 8 == 0, "latent and rope widths must be multiples of 8");
  static_assert(BN % 32 == 0, "key tile must be a multiple of 32");
  static_assert(VOFF + DVB * 32 <= STRIDE, "transpose reads must stay inside a tile row");
  static_assert(DQKP % 32 == 0, "the swizzle permutes chunks within aligned groups of four");
  static_assert(!DENSE || (DR == 0 && DC % 32 == 0 && OW % 32 == 0), "per-head tile layout");
  static_assert(BN * CPR % 64 == 0, "a tile is a whole number of 64-lane loads");
  static constexpr bool SW16 = DENSE && CPR % 16 == 0;
  // chunk position of logical chunk c in row r (an involution: it also maps back)
  __device__ static constexpr int pos(int r, int c) {
    return SW16 ? ((c & ~15) | ((c ^ (((r & 3) << 2) | ((r >> 2) & 3))) & 15))
                : ((c & ~3) | ((c ^ (r >> 2)) & 3));
  }
  // element offset of (row r, column c) inside a tile
  __device__ static constexpr int at(int r, int c) {
    return r * STRIDE + pos(r, c >> 3) * 8 + (c & 7);
  }
};

template <int DC, int DR, int QB, int NW, int BN, int WPC, bool DENSE = false, int DVW = 0,
          int VS = 1>
__global__ __launch_bounds__(NW * 64, WPC) void latent_attend_kernel(const AttendArgs a) {
  using C = AttCfg<DC, DR, QB, NW, BN, DENSE, DVW, VS>;
  __shared__ __attribute__((aligned(16))) uint16_t tile[C::NBUF][C::TILE];
  __shared__ __attribute__((aligned(16))) float resc[NW][64 * 16];
  // pair split: partial score tiles, [tile parity][wave][4 chunks][64 lanes][4]
  __shared__ __attribute__((aligned(16))) float xch[VS > 1 ? 2 : 1][VS > 1 ? NW : 1][64 * 16];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, l32 = lane & 31;
  // query rows per batch element: (token, head) pairs, head-minor (latent); (head, token)
  // pairs with every head padded to whole row blocks (dense: a row block is one head's)
  const int rows_b = DENSE ? a.n_heads * a.nq_pad : a.geo.q_count * a.n_heads;
  if (!DENSE) VMLA_STAMP(a, kStampAttend, 0);
  int stamp_step = 0;  // steps taken by this workgroup (used by the phase stamps only)
  int stamp_seg = 0;   // segments finished by this workgroup (the same)

  // This workgroup's share of the (batch, row block, key tile) units; each maximal run of
  // tiles of one row block is a segment with its own partial result.
  const int64_t U = a.units;
  const int G = a.n_wg, T = a.tiles_per_row;
  int64_t u_begin = (int64_t)blockIdx.x * U / G, u_end = (int64_t)(blockIdx.x + 1) * U / G;
  // Weighted split: the per-XCD weights the partition state holds (set by bal_prep_kernel for an
  // adaptive call, left as they are for a frozen one); an adaptive call records each
  // workgroup's duration for the next one.
  uint32_t bw[8];
  uint64_t bal_t0 = 0;
  if (a.bal_on) {
    bal_weights(a.bal_state, G, bw);
#pragma unroll
    for (int x = 0; x < 8; ++x) bw[x] = __builtin_amdgcn_readfirstlane(bw[x]);
    u_begin = bal_start(bw, G, U, blockIdx.x);
    u_end = bal_start(bw, G, U, blockIdx.x + 1);
    if (a.bal_rec) bal_t0 = __builtin_amdgcn_s_memrealtime();
  }
  // Segments are taken last to first: a workgroup's last segment is the head of a row block
  // (keys from 0) and its first the tail of another, so in this order every workgroup walks the
  // keys at about the same position at the same time (all ranges have the same length), and
  // the workgroups of one XCD find most tiles already in its L2.
  for (int64_t u = u_end; u > u_begin;) {
  const int64_t rbg = (u - 1) / T;
  const int64_t seg_lo = max(u_begin, rbg * T);
  const int kt0 = (int)(seg_lo - rbg * T);
  const int kt1 = (int)(u - rbg * T);
  u = seg_lo;
  const int b = (int)(rbg / a.row_blocks), rb = (int)(rbg % a.row_blocks);
  const int split = (int)blockIdx.x - (a.bal_on ? bal_owner(bw, G, U, rbg * T) : attend_owner(rbg * T, U, G));
  const int vpar = VS > 1 ? wave % VS : 0;  // column half of this wave (pair split)
  const int row0 = rb * C::ROWS + wave / VS * QB * 32;
  const int key_begin = kt0 * BN;
  const int key_end = min(a.n_valid, kt1 * BN);
  const int n_tiles = kt1 - kt0;
  __syncthreads();  // the previous segment's LDS tiles are no longer read

  const u32x4 zero = {0, 0, 0, 0};

  // Direct global-to-LDS staging. Load instruction j (of NDMA per tile) fills the 64 chunk
  // slots 64 j .. 64 j + 63 of a tile; this wave issues j = wave + NW i. Each lane fetches the
  // chunk whose swizzled slot is its own: row r = slot / CPR, logical chunk = physical chunk
  // with the swizzle undone (c_kv chunks, then k_r chunks, then padding that reads k_r data and
  // meets the zero padding of q_cat). Rows at or past key_end are clamped to key_end - 1, so
  // every read stays inside the valid ring and every staged value is finite; their scores
  // are masked below.
  int dma_row[C::DMA_PER_WAVE];
  const uint16_t* dma_src[C::DMA_PER_WAVE];
  bool dma_kr[C::DMA_PER_WAVE];
  if constexpr (DENSE) {
    // one head's [K | V] rows: ring [B][ring_tokens][H][2 * head width]
    const int h = rb / (a.row_blocks / a.n_heads);
    const uint16_t* kv_base = a.kv + ((size_t)b * a.geo.ring_tokens * a.n_heads + h) * C::STRIDE;
#pragma unroll
    for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
      const int j = wave + NW * i;
      const int slot = (j < C::NDMA ? j : 0) * 64 + lane;
      const int r = slot / C::CPR;
      dma_row[i] = r;
      dma_kr[i] = false;
      dma_src[i] = kv_base + C::pos(r, slot % C::CPR) * 8;
    }
  } else {
    const uint16_t* c_base = a.c_kv + (size_t)b * a.geo.ring_tokens * DC;
    const uint16_t* r_base = a.k_r + (size_t)b * a.geo.ring_tokens * DR;
#pragma unroll
    for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
      const int j = wave + NW * i;
      const int slot = (j < C::NDMA ? j : 0) * 64 + lane;
      const int r = slot / C::CPR, pcn = slot % C::CPR;
      const int lc = (pcn & ~3) | ((pcn & 3) ^ ((r >> 2) & 3));
      dma_row[i] = r;
      dma_kr[i] = lc >= C::OCT_C;
      dma_src[i] = lc < C::OCT_C ? c_base + lc * 8
                                 : r_base + (lc < C::OCT_C + C::OCT_R ? (lc - C::OCT_C) * 8 : 0);
    }
  }


  // queries of this wave, B-operand layout: lane holds row l32, dims ks*16 + 8g .. +8 (of the
  // wave's NSH score steps, which start at step vpar * NSH)
  bf16x8 q[QB][C::NSH];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = row0 + qb * 32 + l32;
    const uint16_t* src = a.qcat + ((size_t)b * rows_b + (r < rows_b ? r : 0)) * C::DQKP +
                          vpar * C::NSH * 16;
#pragma unroll
    for (int ks = 0; ks < C::NSH; ++ks)
      q[qb][ks] = as_bf16x8(r < rows_b ? ldg16(src + ks * 16 + 8 * g) : zero);
  }

  f32x16 o[QB][C::DVBW];
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = kNegInf;
    l_run[qb] = 0.f;
#pragma unroll
    for (int d = 0; d < C::DVBW; ++d) o[qb][d] = f32x16{};
  }

  auto dma_tile = [&](int k0, uint16_t* buf) {
    const uint32_t base = lds_addr(buf);
#pragma unroll
    for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
      const int j = wave + NW * i;
      if (C::NDMA % NW == 0 || j < C::NDMA) {
        const int key = min(k0 + dma_row[i], key_end - 1);
        const uint16_t* src =
            dma_src[i] + (size_t)key * (DENSE ? a.n_heads * C::STRIDE : (dma_kr[i] ? DR : DC));
        lds_dma16(src, __builtin_amdgcn_readfirstlane(base + 1024u * j));
      }
    }
  };
  // K operand of step ks: row l32 (+32 kb), chunk 2 ks + g, i.e. C::at(). Latent: the XOR folded
  // into one of two per-lane bases (ks even / odd) so that ks and kb become immediate offsets;
  // dense: one offset per step (its 4-bit XOR reaches every chunk of a group).
  // With the pair split, local step ks is global step vpar * NSH + ks, whose parity picks the base.
  const int hk = (l32 >> 2) & 3;
  const int koff_ev = l32 * C::STRIDE + ((g ^ hk) << 3);
  const int koff_od = l32 * C::STRIDE + (((2 + g) ^ hk) << 3) - 16;
  const bool kflip = (vpar * C::NSH) & 1;
  const int koff_e = (kflip ? koff_od : koff_ev) + vpar * C::NSH * 16;
  const int koff_o = (kflip ? koff_ev : koff_od) + vpar * C::NSH * 16;
  int koff_d[DENSE ? C::KSTEPS : 1];
  if constexpr (DENSE) {
#pragma unroll
    for (int ks = 0; ks < C::KSTEPS; ++ks) koff_d[ks] = C::at(l32, ks * 16 + 8 * g);
  }
  auto koff = [&](int ks) {
    if constexpr (DENSE) return koff_d[ks];
    else return ((ks & 1) ? koff_o : koff_e) + ks * 16;
  };
  // S^T for one tile, the query blocks sharing each K operand read
  auto scores = [&](const uint16_t* buf, f32x16 (&s)[QB][C::KB]) {
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) s[qb][kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < C::NSH; ++ks) {
        const bf16x8 k = as_bf16x8(*reinterpret_cast<const u32x4*>(
            &buf[koff(ks) + kb * 32 * C::STRIDE]));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[qb][kb] = mfma32(k, q[qb][ks], s[qb][kb]);
      }
    }
  };
  // Pair split: publish this wave's partial scores of tile parity `par` (before a barrier), then
  // (after it) add the partner's. Chunk j of lane l sits at (64 j + l) * 4 floats, so every
  // 16-byte access of a wave covers consecutive addresses.
  auto xch_put = [&](int par, const f32x16 (&s)[QB][C::KB]) {
    if constexpr (VS > 1) {
      float* dst = &xch[par][wave][lane * 4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<f32x4*>(dst + 256 * j) =
            f32x4{s[0][0][4 * j], s[0][0][4 * j + 1], s[0][0][4 * j + 2], s[0][0][4 * j + 3]};
    }
  };
  auto xch_add = [&](int par, f32x16 (&s)[QB][C::KB]) {
    if constexpr (VS > 1) {
      const float* src = &xch[par][wave ^ 1][lane * 4];
      // vpar 0 computes mine + partner's and vpar 1 partner's + mine: the same sum either way
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(src + 256 * j);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          s[0][0][4 * j + i] = vpar == 0 ? s[0][0][4 * j + i] + v[i] : v[i] + s[0][0][4 * j + i];
      }
    }
  };
  // keys at or past key_end get -inf
  auto mask_tail = [&](int kbase, f32x16 (&s)[QB][C::KB]) {
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool dead = kbase + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3) >= key_end;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[qb][kb][r] = dead ? kNegInf : s[qb][kb][r];
      }
  };
  // Raise the running max where the scores `s` would exceed it by more than kLazyMax. Each lane
  // sees half of its row's keys; growth on either half sends the wave through the rare path,
  // where the two halves agree on the new max and the accumulators are rescaled through this
  // wave's LDS slot (no VALU instruction ever touches them, so they stay in accumulation
  // registers).
  float own_max[QB];
  auto own_max_of = [&](const f32x16 (&s)[QB][C::KB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      // a tree of three-input maxima (depth 3) rather than a chain of 16
      float m = kNegInf;
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb) {
        const f32x16& v = s[qb][kb];
        const float a0 = fmaxf(fmaxf(v[0], v[1]), v[2]), a1 = fmaxf(fmaxf(v[3], v[4]), v[5]);
        const float a2 = fmaxf(fmaxf(v[6], v[7]), v[8]), a3 = fmaxf(fmaxf(v[9], v[10]), v[11]);
        const float a4 = fmaxf(fmaxf(v[12], v[13]), v[14]);
        m = fmaxf(m, fmaxf(fmaxf(fmaxf(a0, a1), a2), fmaxf(fmaxf(a3, a4), v[15])));
      }
      own_max[qb] = m;
    }
  };
  auto raise_max_if_needed = [&]() {
    bool grow = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) grow |= own_max[qb] > m_run[qb] + kLazyMax;
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {
      f32x16* slot = reinterpret_cast<f32x16*>(&resc[wave][lane * 16]);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float m_new = fmaxf(m_run[qb], half_swap_max(own_max[qb]));
        const float alpha = fast_exp2(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int d = 0; d < C::DVBW; ++d) {
          *slot = o[qb][d];
          asm volatile("" ::: "memory");
          f32x16 tmp = *slot;
          tmp *= alpha;
          *slot = tmp;
          asm volatile("" ::: "memory");
          o[qb][d] = *slot;
        }
      }
    }
  };

  // V^T transpose reads: lane addresses row 4g + tr_row (+8 for the upper half, +16 kk) and
  // column tr_col (+32 d); rows 4g.. have swizzle g, rows 4g+8.. have g+2, for every kk
  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  // (the latent swizzle permutes chunks within 32-column groups, so a whole number of 32-column
  // blocks is a plain offset: this wave's value half starts vpar * DVBW blocks in)
  const int vofs_lo = C::at(4 * g + tr_row, C::VOFF + tr_col) + vpar * C::DVBW * 32;
  const int vofs_hi = C::at(4 * g + tr_row + 8, C::VOFF + tr_col) + vpar * C::DVBW * 32;
  // dense: the 4-bit XOR also permutes the 32-column blocks d, so one offset per (half, d)
  int vofs_d[2][DENSE ? C::DVB : 1];
  if constexpr (DENSE) {
#pragma unroll
    for (int d = 0; d < C::DVB; ++d) {
      vofs_d[0][d] = C::at(4 * g + tr_row, C::VOFF + tr_col + 32 * d);
      vofs_d[1][d] = C::at(4 * g + tr_row + 8, C::VOFF + tr_col + 32 * d);
    }
  }

  // One pipelined step. s_cur holds tile t's scores, already masked, with m_run high enough
  // for them. Block A: scores of tile t+1 (MFMA) and tile t's exponentials (VALU). Block B: PV
  // of tile t (MFMA) and staging of tile t+2. After the barrier: masking and max of tile t+1.
  auto step = [&](int t, f32x16 (&s_cur)[QB][C::KB], f32x16 (&s_nxt)[QB][C::KB],
                  const uint16_t* cur, const uint16_t* nxt, uint16_t* stg) {
    const int kbase = key_begin + t * BN;

    // Work of one step: QK = scores of tile t+1 (14 MFMAs, one LDS read each), SM = the
    // softmax of tile t (exp2, bf16 rounding, row sums; VALU), PV = O += V^T P^T of tile t
    // (12 MFMAs, two LDS transpose reads each). They run as one fenced instruction stream of
    // slots: slot i holds QK MFMA i, then (for the first four slots) a quarter of SM, then PV
    // MFMA i - 2, with every K read issued two slots ahead and every V^T read one slot ahead,
    // so the wave's LDS traffic and VALU work are spread evenly under its MFMAs.
    dma_tile(kbase + 2 * BN, stg);  // buffer of tile t-1, free since the last barrier
    static_assert(C::KB == 1, "the step is laid out for 32-key tiles");
    constexpr int NS = C::NSH;
    constexpr int NPV = 2 * C::DVBW;  // PV operand reads per tile (each feeds QB MFMAs)
    constexpr int NSLOT = NS > NPV + 2 ? NS : NPV + 2;
    constexpr int NSM = NS < 4 ? NS : 4;  // slots carrying the softmax; pairs 0-3 precede PV
    auto kread = [&](int ks) {
      return as_bf16x8(*reinterpret_cast<const u32x4*>(&nxt[koff(ks)]));
    };
    const lds_u16* vlo = as_lds(cur) + vofs_lo;
    const lds_u16* vhi = as_lds(cur) + vofs_hi;
    auto vread = [&](int j) {  // A operand of PV MFMA j: kk = j / DVBW, d = j % DVBW
      const int kk = j / C::DVBW, d = j % C::DVBW;
      if constexpr (DENSE)
        return join_bf16x8(lds_read_tr(as_lds(cur) + vofs_d[0][d] + kk * 16 * C::STRIDE),
                           lds_read_tr(as_lds(cur) + vofs_d[1][d] + kk * 16 * C::STRIDE));
      else
        return join_bf16x8(lds_read_tr(vlo + kk * 16 * C::STRIDE + d * 32),
                           lds_read_tr(vhi + kk * 16 * C::STRIDE + d * 32));
    };
    // The row sum is taken over the bf16-rounded probabilities, the same values the PV MFMA
    // multiplies, so numerator and denominator see identical weights.
    uint32_t pk[QB][8];
    float lsum[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) lsum[qb] = l_run[qb];
    auto sm_pair = [&](int qb, int p) {
      const f32x2 e = {fast_exp2(s_cur[qb][0][2 * p] - m_run[qb]),
                       fast_exp2(s_cur[qb][0][2 * p + 1] - m_run[qb])};
      const bf16x2 h = __builtin_convertvector(e, bf16x2);
      lsum[qb] = __builtin_amdgcn_fdot2_f32_bf16(h, kOnesBf16x2, lsum[qb], false);
      pk[qb][p] = __builtin_bit_cast(uint32_t, h);
    };
    f32x16 acc[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) acc[qb] = f32x16{};
    bf16x8 kq[3], vq[2];
    kq[0] = kread(0);
    if (NS > 1) kq[1] = kread(1);
#pragma unroll
    for (int ks = 0; ks < NSLOT; ++ks) {
      if (ks + 2 < NS) kq[(ks + 2) % 3] = kread(ks + 2);
      const int j = ks - 2;  // PV operand of this slot
      if (j + 1 >= 0 && j + 1 < NPV) vq[(j + 1) & 1] = vread(j + 1);
      // Issue priority 1 for the first half of the slots, 0 for the second: of the two waves
      // sharing a SIMD's matrix pipe, the one that is behind wins it more often, so they
      // finish their streams closer together (the older wave otherwise takes the pipe first
      // and the younger one ends the step alone, at a lower MFMA rate).
      __builtin_amdgcn_sched_barrier(0);
      if (ks == 0) __builtin_amdgcn_s_setprio(1);
      if (ks == NSLOT / 2) __builtin_amdgcn_s_setprio(0);
      if (ks < NS) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) acc[qb] = mfma32(kq[ks % 3], q[qb][ks], acc[qb]);
      }
      if (ks < NSM) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int p = ks * 8 / NSM; p < (ks + 1) * 8 / NSM; ++p) sm_pair(qb, p);
      }
      if (j >= 0 && j < NPV) {
        const int kk = j / C::DVBW, d = j % C::DVBW;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          const bf16x8 pb = as_bf16x8(kk == 0 ? u32x4{pk[qb][0], pk[qb][1], pk[qb][2], pk[qb][3]}
                                              : u32x4{pk[qb][4], pk[qb][5], pk[qb][6], pk[qb][7]});
          o[qb][d] = mfma32(vq[j & 1], pb, o[qb][d]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      s_nxt[qb][0] = acc[qb];
      l_run[qb] = lsum[qb];
    }
    xch_put((t + 1) & 1, s_nxt);
    // phase stamps: the stream's end is read here and stored after the barrier, so that the
    // wait below has no stamp store to drain
    const bool stamped = !DENSE && stamp_step >= 200 && stamp_step < 204;
    const uint64_t stream_end = stamped ? VMLA_STAMP_NOW() : 0;
    wait_vmcnt<0>();  // this wave's part of tile t+2 is in LDS
    __syncthreads();
    if (stamped) {
      VMLA_STAMP(a, kStampAttend, 3 + 2 * (stamp_step - 200));
      VMLA_STAMP_AT(a, kStampAttend, 2 + 2 * (stamp_step - 200), stream_end);
    }
    ++stamp_step;
    xch_add((t + 1) & 1, s_nxt);
    if (kbase + 2 * BN > key_end) mask_tail(kbase + BN, s_nxt);  // only near the split's end
    own_max_of(s_nxt);
    raise_max_if_needed();
  };

  if (n_tiles > 0) {
    dma_tile(key_begin, tile[0]);
    dma_tile(key_begin + BN, tile[1]);
  }
  wait_vmcnt<0>();
  __syncthreads();
  if (!DENSE && stamp_step == 0) VMLA_STAMP(a, kStampAttend, 1);
  if (!DENSE && stamp_seg == 1) VMLA_STAMP(a, kStampAttend, 14);

  f32x16 s_a[QB][C::KB], s_b[QB][C::KB];
  if (n_tiles > 0) scores(tile[0], s_a);
  if constexpr (VS > 1) {
    if (n_tiles > 0) xch_put(0, s_a);
    __syncthreads();
    if (n_tiles > 0) xch_add(0, s_a);
  }
  if (n_tiles > 0) {
    if (key_begin + BN > key_end) mask_tail(key_begin, s_a);
    own_max_of(s_a);
    raise_max_if_needed();  // sets the running max from the first tile
  }
  // tile t lives in buffer t mod 3; the three buffer pointers rotate with the tiles
  uint16_t *pc = tile[0], *pn = tile[1], *ps = tile[2];
  int t = 0;
  for (; t + 1 < n_tiles; t += 2) {
    step(t, s_a, s_b, pc, pn, ps);
    step(t + 1, s_b, s_a, pn, ps, pc);
    uint16_t* tmp = pc;
    pc = ps;
    ps = pn;
    pn = tmp;
  }
  if (t < n_tiles) step(t, s_a, s_b, pc, pn, ps);
  if (!DENSE) VMLA_STAMP(a, kStampAttend, 10);  // the segment processed last keeps its stamp
  if (!DENSE && stamp_seg == 0) VMLA_STAMP(a, kStampAttend, 12);

  // ---- write unnormalized O_lat and (max, sum) of this split -------------------------------
  const size_t total_rows = (size_t)a.batch * rows_b;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l_tot = half_swap_sum(l_run[qb]);
    const int r = row0 + qb * 32 + l32;
    if (r >= rows_b) continue;
    const size_t grow_i = (size_t)b * rows_b + r;
    float* op = a.o_part + ((size_t)split * total_rows + grow_i) * C::OW;
#pragma unroll
    for (int d = 0; d < C::DVBW; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = (vpar * C::DVBW + d) * 32 + 8 * i + 4 * g;
        if (c < C::OW) {
          const f32x4 v = {o[qb][d][4 * i], o[qb][d][4 * i + 1], o[qb][d][4 * i + 2], o[qb][d][4 * i + 3]};
          *reinterpret_cast<f32x4*>(op + c) = v;
        }
      }
    if (g == 0 && vpar == 0) {
      float* ml = a.ml_part + ((size_t)split * total_rows + grow_i) * 2;
      ml[0] = m_run[qb];
      ml[1] = l_tot;
    }
  }
  if (!DENSE && stamp_seg == 0) VMLA_STAMP(a, kStampAttend, 13);
  ++stamp_seg;
  }  // segments
  if (!DENSE) VMLA_STAMP_DRAINED(a, kStampAttend, 11);
  if (a.bal_rec && tid == 0)
    a.bal_state[kBalHead + blockIdx.x] = (uint32_t)(__builtin_amdgcn_s_memrealtime() - bal_t0);
}

// ---------------------------------------------------------------------------------------------
// out_proj: grid (ceil(Nq / (32 NW)), H, B), NW waves x 32 tokens, one head per workgroup.
// Each wave handles the rows (token n, head h) of its 32 tokens:
//   1. merge coefficients of every row over its key splits s: M = max_s m_s,
//      L = sum_s 2^(m_s - M) l_s, coef_s = 2^(m_s - M) / L, kept in LDS; the first group's
//      split-0 partial rows are already in flight meanwhile
//   2. o_lat = sum_s coef_s O_s, streamed as 16-byte chunks that cover the rows' partial results
//      contiguously, rounded to bf16 into an LDS tile [32][DC]. A lane's chunks go in groups,
//      and the loads of every split of a group (about 24 per lane) are issued before the first
//      is used: the partial results come from HBM, and few loads in flight per wave would
//      leave the kernel bound by their latency
//   3. out^T[v][token] = W_UV_h[v][:] . o_lat[token][:] with MFMA (A = W_UV rows, B = o_lat
//      rows from LDS). Where it fits (WL), W_UV_h is staged in LDS once per workgroup with
//      whole-line loads, issued at the start and stored once the coefficients' loads are back
//      (their latency passes under those); otherwise every wave reads its A operands from
//      global memory.
//   4. the bf16 result is staged through the same LDS tile so that every output row is stored
//      as whole 16-byte chunks.
// The one workgroup barrier follows step 1. Steps 2-4 of a wave touch only its own tile, so a
// wave whose rows have fewer splits runs its MFMAs and stores while the others still load.
// Lanes of tokens past the chunk work on the chunk's last token and store nothing.
// PRE (few-query calls, whose few row blocks are split over many workgroups each): steps 1 and
// 2 are done beforehand by latent_merge_kernel, which runs one thread per (row, 8 columns) over
// every row at once and leaves the merged bf16 o_lat rows [row][DC] in the q_cat area; the
// kernel then copies them into its tile and applies W_UV_h.
// ---------------------------------------------------------------------------------------------
constexpr int kMergeSplits = 4;

template <int DC, int NVB>
struct OutProjShape {
  static constexpr int DV = NVB * 32;
  static constexpr int LS = (DC > DV ? DC : DV) + 8;  // LDS row stride (elements); +16 B per row
  static constexpr int ROWB = 32 * (4 + 4 * kMergeSplits);  // per-wave row scalars
  static constexpr int BUDGET = 160 * 1024 - 512;
  static constexpr int need(int nw, bool wl) { return nw * (32 * LS * 2 + ROWB) + (wl ? DV * LS * 2 : 0); }
  // the most waves per workgroup (8, else 4) that fit with W_UV_h in LDS, else 4 reading it
  // from global memory; fewer waves (down to 2) are launched when the grid would otherwise
  // leave most compute units idle
  static constexpr int NW = need(8, true) <= BUDGET ? 8 : 4;
  static constexpr bool WL = need(NW, true) <= BUDGET;
  static constexpr bool WL4 = need(4, true) <= BUDGET;
  static constexpr bool WL2 = need(2, true) <= BUDGET;
};

template <int DC, int NVB, int NW, bool WL, bool PRE>
__global__ __launch_bounds__(NW * 64) void out_proj_kernel(const AttendArgs a) {
  constexpr int KS = DC / 16;
  constexpr int DV = NVB * 32;
  constexpr int LS = OutProjShape<DC, NVB>::LS;
  constexpr int CH = DC / 4;                   // fp32 chunks of 16 B per partial row
  constexpr int NT = NW * 64;
  static_assert((32 * CH) % 64 == 0 && (32 * DV / 8) % 64 == 0, "whole 64-lane passes");
  __shared__ __attribute__((aligned(16))) uint16_t tileo[NW][32 * LS];
  __shared__ __attribute__((aligned(16))) uint16_t wlds[WL ? DV * LS : 8];
  __shared__ float row_coef[NW][32][kMergeSplits];
  __shared__ int row_ns[NW][32];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, l32 = lane & 31;
  const int h = blockIdx.y, b = blockIdx.z;
  const int H = a.n_heads, Nq = a.geo.q_count;
  const int n0 = blockIdx.x * (NW * 32) + wave * 32;
  const size_t total_rows = (size_t)a.batch * Nq * H;
  auto row_of = [&](int t) {  // global row of the wave's token t
    const int n = min(n0 + t, Nq - 1);
    return ((size_t)b * Nq + n) * H + h;
  };
  uint16_t* tw = tileo[wave];
  const uint16_t* w = a.w_uv + (size_t)h * DV * DC;
  VMLA_STAMP(a, kStampOutProj, 0);

  // 0. W_UV_h [DV][DC] for LDS: every load of this thread issued now, stored once the
  //    coefficients' loads are back
  constexpr int WCPR = DC / 8, WPER = WL ? (DV * WCPR + NT - 1) / NT : 1;
  u32x4 wv[WPER];
  if constexpr (WL) {
#pragma unroll
    for (int i = 0; i < WPER; ++i) {
      const int c = tid + NT * i;
      if (c < DV * WCPR) wv[i] = ldg16(w + (size_t)(c / WCPR) * DC + (c % WCPR) * 8);
    }
  }

  // merge helpers (calls that are not merged beforehand): every row has at most kMergeSplits
  // splits, since calls with more are merged beforehand
  constexpr int NI = 32 * CH / 64;            // 16-byte chunks of the wave's 32 rows per lane
  // chunks per group for a wave whose rows have up to ns splits: the loads of every split of a
  // group are in flight together, about 24 per lane
  constexpr auto group = [](int ns) { int g = 24 / ns < NI ? 24 / ns : NI; while (NI % g) --g; return g; };
  constexpr int NP = group(kMergeSplits);     // split-0 chunks loaded before the coefficients
  auto part = [&](int s, int i) {             // split s's partial of this lane's chunk i
    const int q = i * 64 + lane, t = q / CH, k = q % CH;
    return reinterpret_cast<const f32x4*>(a.o_part + ((size_t)s * total_rows + row_of(t)) * DC + 4 * k);
  };
  f32x4 v0[NP];
  int nsw = 1;                                // the wave's largest split count (uniform)

  if constexpr (PRE) {
    // the merged rows, 16-byte chunks, coalesced
    constexpr int C8 = DC / 8;
#pragma unroll 4
    for (int it = 0; it < 32 * C8 / 64; ++it) {
      const int q = it * 64 + lane;
      const int t = q / C8, k = q % C8;
      *reinterpret_cast<u32x4*>(&tw[t * LS + 8 * k]) = ldg16(a.qcat + row_of(t) * DC + 8 * k);
    }
  } else {
  // 1. every row has a split 0: the first group's loads go out before the coefficients are known
#pragma unroll
  for (int i = 0; i < NP; ++i) v0[i] = *part(0, i);
  // merge coefficients per row (lanes 0..31, one row each): M = max_s m_s, L = sum_s 2^(m_s - M) l_s
  const size_t row = row_of(lane & 31);
  const int64_t rbg = (int64_t)b * a.row_blocks + (int)((row - (size_t)b * Nq * H) / a.att_rows);
  const int ns = attend_split_count(a, rbg);
#pragma unroll
  for (int s = 1; s < kMergeSplits; ++s) nsw += __ballot(ns > s) != 0;
  if (lane < 32) {
    f32x2 ml[kMergeSplits];
#pragma unroll
    for (int s = 0; s < kMergeSplits; ++s)
      ml[s] = s < ns ? *reinterpret_cast<const f32x2*>(a.ml_part + ((size_t)s * total_rows + row) * 2)
                     : f32x2{kNegInf, 0.f};
    float M = kNegInf;
#pragma unroll
    for (int s = 0; s < kMergeSplits; ++s) M = fmaxf(M, ml[s][0]);
    float L = 0.f;
#pragma unroll
    for (int s = 0; s < kMergeSplits; ++s)
      if (s < ns) L += fast_exp2(ml[s][0] - M) * ml[s][1];
    const float il = 1.f / L;
#pragma unroll
    for (int s = 0; s < kMergeSplits; ++s)
      row_coef[wave][lane][s] = s < ns ? fast_exp2(ml[s][0] - M) * il : 0.f;
    row_ns[wave][lane] = ns;
  }
  }  // coefficients in this kernel
  if constexpr (WL) {
#pragma unroll
    for (int i = 0; i < WPER; ++i) {
      const int c = tid + NT * i;
      if (c < DV * WCPR) *reinterpret_cast<u32x4*>(&wlds[(c / WCPR) * LS + (c % WCPR) * 8]) = wv[i];
    }
  }
  __syncthreads();  // the W_UV_h tile (WL), the coefficient tables or (PRE) the copied rows
  VMLA_STAMP(a, kStampOutProj, 1);
  // From here on each wave works on its own LDS tile only. The LDS operations of one wave take
  // effect in program order, so the steps below need no workgroup barrier; wave_order() keeps
  // the compiler from moving LDS accesses across a step boundary.
  auto wave_order = [] {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  if constexpr (!PRE) {
  // 2. o_lat = sum_s coef_s O_s per group of chunks, rounded to bf16 into the LDS tile. NS is
  // the wave's largest split count; a row with fewer splits reads its last one again (the same
  // lines, from cache) and weighs it by a zero coefficient, so the loads need no per-lane
  // branches.
  auto merge = [&](auto nsc) {
    constexpr int NS = decltype(nsc)::value, NG = group(NS);
#pragma unroll
    for (int g = 0; g < NI / NG; ++g) {
      f32x4 u[NS][NG];
#pragma unroll
      for (int i = 0; i < NG; ++i) u[0][i] = g * NG + i < NP ? v0[g * NG + i] : *part(0, g * NG + i);
#pragma unroll
      for (int s = 1; s < NS; ++s)
#pragma unroll
        for (int i = 0; i < NG; ++i) {
          const int t = ((g * NG + i) * 64 + lane) / CH;
          u[s][i] = *part(min(s, row_ns[wave][t] - 1), g * NG + i);
        }
#pragma unroll
      for (int i = 0; i < NG; ++i) {
        const int q = (g * NG + i) * 64 + lane, t = q / CH, k = q % CH;
        f32x4 acc = row_coef[wave][t][0] * u[0][i];
#pragma unroll
        for (int s = 1; s < NS; ++s) acc += row_coef[wave][t][s] * u[s][i];
        *reinterpret_cast<bf16x4*>(&tw[t * LS + 4 * k]) = to_bf16x4(acc);
      }
    }
  };
  static_assert(kMergeSplits == 4, "one case per split count");
  switch (nsw) {
    case 1: merge(std::integral_constant<int, 1>{}); break;
    case 2: merge(std::integral_constant<int, 2>{}); break;
    case 3: merge(std::integral_constant<int, 3>{}); break;
    default: merge(std::integral_constant<int, 4>{}); break;
  }
  }  // merge in this kernel
  wave_order();  // the wave's o_lat tile is complete
  VMLA_STAMP(a, kStampOutProj, 2);

  // 3. out^T = W_UV_h o_lat^T
  f32x16 acc[NVB];
#pragma unroll
  for (int vb = 0; vb < NVB; ++vb) acc[vb] = f32x16{};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const bf16x8 bo = as_bf16x8(*reinterpret_cast<const u32x4*>(&tw[l32 * LS + ks * 16 + 8 * g]));
#pragma unroll
    for (int vb = 0; vb < NVB; ++vb) {
      const bf16x8 aw = WL ? as_bf16x8(*reinterpret_cast<const u32x4*>(&wlds[(vb * 32 + l32) * LS + ks * 16 + 8 * g]))
                           : as_bf16x8(ldg16(w + (size_t)(vb * 32 + l32) * DC + ks * 16 + 8 * g));
      acc[vb] = mfma32(aw, bo, acc[vb]);
    }
  }
  wave_order();  // every lane of the wave is done reading its o_lat tile
  VMLA_STAMP(a, kStampOutProj, 3);

  // 4. stage the bf16 output rows and store them whole
#pragma unroll
  for (int vb = 0; vb < NVB; ++vb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 v = {acc[vb][4 * i], acc[vb][4 * i + 1], acc[vb][4 * i + 2], acc[vb][4 * i + 3]};
      *reinterpret_cast<bf16x4*>(&tw[l32 * LS + vb * 32 + 8 * i + 4 * g]) = to_bf16x4(v);
    }
  wave_order();
  VMLA_STAMP(a, kStampOutProj, 4);
#pragma unroll
  for (int it = 0; it < 32 * DV / 8 / 64; ++it) {
    const int q = it * 64 + lane;
    const int t = q / (DV / 8), k = q % (DV / 8);
    if (n0 + t < Nq)
      *reinterpret_cast<u32x4*>(a.out + row_of(t) * DV + 8 * k) =
          *reinterpret_cast<const u32x4*>(&tw[t * LS + 8 * k]);
  }
  VMLA_STAMP_DRAINED(a, kStampOutProj, 5);
}

// Tile shapes per supported (d_c, d_rope).
template <int DC, int DR> struct AttShape;
// WPC = resident workgroups per CU (the grid is WPC workgroups per CU). Two 4-wave workgroups
// per CU measured 6% slower than one 8-wave workgroup at the Wan shape.
template <> struct AttShape<192, 32> { static constexpr int QB = 1, NW = 8, BN = 32, WPC = 1, VS = 1; };
template <> struct AttShape<16, 8> { static constexpr int QB = 1, NW = 4, BN = 32, WPC = 1, VS = 1; };
// the latent widths of the paper's d_c sweep (Table 5), with the same 32-wide RoPE key
template <> struct AttShape<64, 32> { static constexpr int QB = 1, NW = 8, BN = 32, WPC = 1, VS = 1; };
template <> struct AttShape<128, 32> { static constexpr int QB = 1, NW = 8, BN = 32, WPC = 1, VS = 1; };
// d_c = 256: 32 rows x 256 fp32 accumulators per wave need one wave per SIMD (8 waves spill)
template <> struct AttShape<256, 32> { static constexpr int QB = 1, NW = 4, BN = 32, WPC = 1, VS = 1; };
// d_c = 512: wave pairs split the score contraction and the value columns (pair split), one
// wave per SIMD
template <> struct AttShape<512, 32> { static constexpr int QB = 1, NW = 4, BN = 32, WPC = 1, VS = 2; };

// Every (d_c, d_rope) the latent path is instantiated for.
#define VMLA_LATENT_SHAPES(X) X(192, 32) X(16, 8) X(64, 32) X(128, 32) X(256, 32) X(512, 32)

template <int DC, int DR>
hipError_t launch_attend_t(const AttendArgs& a, hipStream_t s) {
  using S = AttShape<DC, DR>;
  using C = AttCfg<DC, DR, S::QB, S::NW, S::BN, false, 0, S::VS>;
  const dim3 grid(a.n_wg);
  hipLaunchKernelGGL((latent_attend_kernel<DC, DR, S::QB, S::NW, S::BN, S::WPC, false, 0, S::VS>),
                     grid, dim3(C::NT), 0, s, a);
  return hipGetLastError();
}

// Dense comparator: one head of 128 channels per row block, K and V rows interleaved per head.
using DenseShape = AttShape<192, 32>;  // same wave count, tile and occupancy as the latent kernel
constexpr int kDenseHead = 128;
using DenseCfg = AttCfg<kDenseHead, 0, DenseShape::QB, DenseShape::NW, DenseShape::BN, true>;

}  // namespace

bool dense_attend_supported(int d_head) { return d_head == kDenseHead; }
int dense_attend_rows_per_block() { return DenseCfg::ROWS; }
int dense_attend_keys_per_tile() { return DenseShape::BN; }

hipError_t launch_dense_attend(const AttendArgs& a, hipStream_t s) {
  if (a.d_v != kDenseHead) return hipErrorInvalidValue;
  hipLaunchKernelGGL((latent_attend_kernel<kDenseHead, 0, DenseShape::QB, DenseShape::NW,
                                           DenseShape::BN, DenseShape::WPC, true>),
                     dim3(a.n_wg), dim3(DenseCfg::NT), 0, s, a);
  return hipGetLastError();
}

// Materialized form: per-head rows [K_h | V_h] with K_h = [W_UK,h c ; k^R] of width d_nope +
// d_rope (a.dqk_pad) and V_h of width d_v = 128: 128 | 128 is the dense comparator's
// instantiation, 160 | 128 (d_nope 128 + d_rope 32) its own.
bool mat_attend_supported(int d_k, int d_v) {
  return d_v == kDenseHead && (d_k == kDenseHead || d_k == 160);
}

hipError_t launch_mat_attend(const AttendArgs& a, hipStream_t s) {
  if (!mat_attend_supported(a.dqk_pad, a.d_v)) return hipErrorInvalidValue;
  if (a.dqk_pad == kDenseHead) return launch_dense_attend(a, s);
  hipLaunchKernelGGL((latent_attend_kernel<160, 0, DenseShape::QB, DenseShape::NW,
                                           DenseShape::BN, DenseShape::WPC, true, kDenseHead>),
                     dim3(a.n_wg), dim3(DenseCfg::NT), 0, s, a);
  return hipGetLastError();
}

template <int DC, int DR> using ShapeCfg =
    AttCfg<DC, DR, AttShape<DC, DR>::QB, AttShape<DC, DR>::NW, AttShape<DC, DR>::BN, false, 0,
           AttShape<DC, DR>::VS>;

bool latent_attend_supported(int d_c, int d_rope) {
#define X(DC, DR) if (d_c == DC && d_rope == DR) return true;
  VMLA_LATENT_SHAPES(X)
#undef X
  return false;
}

int latent_attend_rows_per_block(int d_c, int d_rope) {
#define X(DC, DR) if (d_c == DC && d_rope == DR) return ShapeCfg<DC, DR>::ROWS;
  VMLA_LATENT_SHAPES(X)
#undef X
  return 0;
}

int latent_attend_keys_per_tile(int d_c, int d_rope) {
#define X(DC, DR) if (d_c == DC && d_rope == DR) return AttShape<DC, DR>::BN;
  VMLA_LATENT_SHAPES(X)
#undef X
  return 0;
}

int latent_attend_wgs_per_cu(int d_c, int d_rope) {
#define X(DC, DR) if (d_c == DC && d_rope == DR) return AttShape<DC, DR>::WPC;
  VMLA_LATENT_SHAPES(X)
#undef X
  return 0;
}

size_t q_absorb_lds_bytes(int d_c, int d_rope, int d_nope) {
#define X(DC, DR)                                                                      \
  if (d_c == DC && d_rope == DR) {                                                     \
    const size_t w = (size_t)d_nope * (AbsorbChunk<DC>::CW + 8);                       \
    const size_t o = AbsorbChunk<DC>::STAGE ? 4 * 32 * ((DC + DR + 15) / 16 * 16 + 8) : 0; \
    return (w > o ? w : o) * 2;                                                        \
  }
  VMLA_LATENT_SHAPES(X)
#undef X
  return 0;
}

hipError_t launch_q_absorb(const AttendArgs& a, hipStream_t s) {
  const dim3 grid((a.geo.q_count + 127) / 128, a.n_heads, a.batch);
  const size_t lds = q_absorb_lds_bytes(a.d_c, a.d_rope, a.d_nope);
#define X(DC, DR)                                                                    \
  if (a.d_c == DC && a.d_rope == DR) {                                               \
    hipLaunchKernelGGL((q_absorb_kernel<DC, DR>), grid, dim3(256), lds, s, a);       \
    return hipGetLastError();                                                        \
  }
  VMLA_LATENT_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

hipError_t launch_rope_window(const AttendArgs& a, hipStream_t s) {
  const int64_t threads = (int64_t)a.n_valid * (a.d_rope / 2);
  hipLaunchKernelGGL(rope_window_kernel, dim3((unsigned)((threads + 255) / 256), a.batch),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_bal_prep(const AttendArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(bal_prep_kernel, dim3(1), dim3(64), 0, s, a.bal_state, a.n_wg);
  return hipGetLastError();
}

hipError_t launch_latent_attend(const AttendArgs& a, hipStream_t s) {
#define X(DC, DR) if (a.d_c == DC && a.d_rope == DR) return launch_attend_t<DC, DR>(a, s);
  VMLA_LATENT_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

int out_proj_cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
    return n;
  return 256;
}

template <int DC, int NVB, bool PRE>
hipError_t launch_out_proj_v(const AttendArgs& a, hipStream_t s) {
  using P = OutProjShape<DC, NVB>;
  // waves per workgroup: the largest of P::NW, 4, 2 whose grid covers at least half of the CUs
  // (four waves with W_UV_h in LDS hold one workgroup per CU, so a grid of more than one
  // workgroup per CU would run in two rounds)
  auto wgs = [&](int nw) { return (int64_t)((a.geo.q_count + 32 * nw - 1) / (32 * nw)) * a.n_heads * a.batch; };
  const int n_cu = out_proj_cu_count();
  int nw = P::NW;
  if (2 * wgs(nw) < n_cu && nw > 4) nw = 4;
  if (2 * wgs(nw) < n_cu && nw > 2) nw = 2;
  const dim3 grid((a.geo.q_count + 32 * nw - 1) / (32 * nw), a.n_heads, a.batch);
  if (nw == P::NW) hipLaunchKernelGGL((out_proj_kernel<DC, NVB, P::NW, P::WL, PRE>), grid, dim3(64 * nw), 0, s, a);
  else if (nw == 4) hipLaunchKernelGGL((out_proj_kernel<DC, NVB, 4, P::WL4, PRE>), grid, dim3(64 * nw), 0, s, a);
  else hipLaunchKernelGGL((out_proj_kernel<DC, NVB, 2, P::WL2, PRE>), grid, dim3(64 * nw), 0, s, a);
  return hipGetLastError();
}

template <int DC, bool PRE>
hipError_t launch_out_proj_t(const AttendArgs& a, hipStream_t s) {
  switch (a.d_v / 32) {
    case 1: return launch_out_proj_v<DC, 1, PRE>(a, s);
    case 2: return launch_out_proj_v<DC, 2, PRE>(a, s);
    case 3: return launch_out_proj_v<DC, 3, PRE>(a, s);
    case 4: return launch_out_proj_v<DC, 4, PRE>(a, s);
    case 5: return launch_out_proj_v<DC, 5, PRE>(a, s);
    case 6: return launch_out_proj_v<DC, 6, PRE>(a, s);
    case 7: return launch_out_proj_v<DC, 7, PRE>(a, s);
    case 8: return launch_out_proj_v<DC, 8, PRE>(a, s);
    default: return hipErrorInvalidValue;
  }
}

bool out_proj_premerged(const AttendArgs& a) { return a.max_seg > kMergeSplits; }

hipError_t launch_out_proj(const AttendArgs& a, hipStream_t s) {
  const bool pre = out_proj_premerged(a);
#define X(DC, DR) \
  if (a.d_c == DC && a.d_rope == DR) \
    return pre ? launch_out_proj_t<DC, true>(a, s) : launch_out_proj_t<DC, false>(a, s);
  VMLA_LATENT_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace vmla
