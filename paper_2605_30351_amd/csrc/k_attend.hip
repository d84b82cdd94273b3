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
#include "vmla_device.h"

namespace vmla {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

// ---------------------------------------------------------------------------------------------
// q_absorb: grid (ceil(Nq/128), H, B), 4 waves, 32 tokens per wave, one head per workgroup.
// out^T[c][token] = W_UK_h^T[c][k] q_nope^T[k][token]; W_UK_h ([d_nope][d_c] row-major) is
// staged in LDS and read transposed with ds_read_b64_tr_b16.
// ---------------------------------------------------------------------------------------------
template <int DC, int DR>
__global__ __launch_bounds__(256) void q_absorb_kernel(const AttendArgs a) {
  constexpr int DCP = (DC + 31) / 32 * 32;
  constexpr int WS = DCP + 8;  // LDS row stride (elements)
  constexpr int DQKP = (DC + DR + 15) / 16 * 16;
  extern __shared__ __attribute__((aligned(16))) uint16_t wuk[];  // [d_nope][WS]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int h = blockIdx.y, b = blockIdx.z;
  const int H = a.n_heads, dn = a.d_nope, Nq = a.geo.chunk_tokens;

  const uint16_t* wsrc = a.w_uk + (size_t)h * dn * DC;
  for (int c = tid; c < dn * (DC / 8); c += 256) {
    const int r = c / (DC / 8), oc = c % (DC / 8);
    *reinterpret_cast<u32x4*>(&wuk[r * WS + oc * 8]) = ldg16(wsrc + (size_t)r * DC + oc * 8);
  }
  __syncthreads();

  const int n = blockIdx.x * 128 + wave * 32 + l32;
  const bool ok = n < Nq;
  const size_t row = ((size_t)b * Nq + (ok ? n : 0)) * H + h;
  const uint16_t* qn = a.q_nope + row * dn;
  uint16_t* dst = a.qcat + row * DQKP;

  // tr-read addressing inside a 16-lane group
  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const u32x4 zero = {0, 0, 0, 0};
#pragma unroll
  for (int cb = 0; cb < DCP / 32; ++cb) {
    f32x16 acc = {};
    for (int ks = 0; ks < dn / 16; ++ks) {
      const int k0 = ks * 16 + 8 * g;
      const i16x4 lo = lds_read_tr(&wuk[(k0 + tr_row) * WS + cb * 32 + tr_col]);
      const i16x4 hi = lds_read_tr(&wuk[(k0 + 4 + tr_row) * WS + cb * 32 + tr_col]);
      const bf16x8 bq = as_bf16x8(ok ? ldg16(qn + k0) : zero);
      acc = mfma32(join_bf16x8(lo, hi), bq, acc);
    }
    if (ok) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = cb * 32 + 8 * i + 4 * g;
        if (c < DC) {
          const f32x4 v = {acc[4 * i] * a.qscale, acc[4 * i + 1] * a.qscale,
                           acc[4 * i + 2] * a.qscale, acc[4 * i + 3] * a.qscale};
          *reinterpret_cast<bf16x4*>(dst + c) = to_bf16x4(v);
        }
      }
    }
  }

  // RoPE part and zero padding: 32 tokens x (DR/2) pairs per wave.
  const int tok0 = blockIdx.x * 128 + wave * 32;
  for (int it = lane; it < 32 * (DR / 2); it += 64) {
    const int t = tok0 + it / (DR / 2), p = it % (DR / 2);
    if (t >= Nq) continue;
    const size_t r = ((size_t)b * Nq + t) * H + h;
    const uint32_t raw = *reinterpret_cast<const uint32_t*>(a.q_r + r * DR + 2 * p);
    float u = bf16_bits_to_f32((uint16_t)(raw & 0xffff)), v = bf16_bits_to_f32((uint16_t)(raw >> 16));
    rope_rotate(a.rope, p, token_pos(a.geo, t), u, v);
    const uint32_t packed =
        (uint32_t)to_bf16_bits(u * a.qscale) | ((uint32_t)to_bf16_bits(v * a.qscale) << 16);
    *reinterpret_cast<uint32_t*>(a.qcat + r * DQKP + DC + 2 * p) = packed;
  }
  if (DQKP > DC + DR) {
    for (int t = tok0 + lane; t < tok0 + 32 && t < Nq; t += 64) {
      const size_t r = ((size_t)b * Nq + t) * H + h;
      for (int c = DC + DR; c < DQKP; ++c) a.qcat[r * DQKP + c] = 0;
    }
  }
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
//   Tiles are fetched with bounds-checked buffer loads whose range ends at the segment's last
//   valid key, so keys past it read as zeros without any branch. The (batch, row block, key
//   tile) units are split evenly over the workgroups (a row block may be shared by two or
//   three of them), so every CU gets the same amount of work.
// ---------------------------------------------------------------------------------------------
constexpr float kLazyMax = 8.0f;
constexpr int kRawBufferWord3 = 0x00020000;  // raw (untyped) buffer access, 32-bit data format

template <int DC, int DR, int QB, int NW, int BN>
struct AttCfg {
  static constexpr int DQK = DC + DR;
  static constexpr int DQKP = (DQK + 15) / 16 * 16;
  static constexpr int KSTEPS = DQKP / 16;
  static constexpr int DVB = (DC + 31) / 32;
  static constexpr int KB = BN / 32;       // 32-key blocks per tile
  static constexpr int STRIDE = DQKP + 8;  // elements; +16 B per row against bank conflicts
  static constexpr int NT = NW * 64;
  static constexpr int ROWS = NW * QB * 32;
  static constexpr int OCT_C = DC / 8, OCT_R = DR / 8;
  static constexpr int CH_C = BN * OCT_C, CH_R = BN * OCT_R;
  static constexpr int CPT_C = (CH_C + NT - 1) / NT;  // c_kv chunks per thread
  static constexpr int CPT_R = (CH_R + NT - 1) / NT;  // k_r chunks per thread
  static constexpr int TILE = BN * STRIDE;
  static constexpr int NBUF = 3;
  static_assert(DC % 8 == 0 && DR % 8 == 0, "latent and rope widths must be multiples of 8");
  static_assert(BN % 32 == 0, "key tile must be a multiple of 32");
  static_assert(DVB * 32 <= STRIDE, "transpose reads must stay inside a tile row");
};

template <int DC, int DR, int QB, int NW, int BN>
__global__ __launch_bounds__(NW * 64, 1) void latent_attend_kernel(const AttendArgs a) {
  using C = AttCfg<DC, DR, QB, NW, BN>;
  __shared__ __attribute__((aligned(16))) uint16_t tile[C::NBUF][C::TILE];
  __shared__ __attribute__((aligned(16))) float resc[NW][64 * 16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int rows_b = a.geo.chunk_tokens * a.n_heads;
  if (C::DQKP > C::DQK) {  // zero the pad columns once; staging never writes them
    for (int r = tid; r < C::NBUF * BN; r += C::NT)
      for (int c = C::DQK; c < C::DQKP; ++c) tile[r / BN][(r % BN) * C::STRIDE + c] = 0;
  }

  // This workgroup's share of the (batch, row block, key tile) units; each maximal run of
  // tiles of one row block is a segment with its own partial result.
  const int64_t U = a.units;
  const int G = a.n_wg, T = a.tiles_per_row;
  const int64_t u_begin = (int64_t)blockIdx.x * U / G, u_end = (int64_t)(blockIdx.x + 1) * U / G;
  for (int64_t u = u_begin; u < u_end;) {
  const int64_t rbg = u / T;
  const int kt0 = (int)(u - rbg * T);
  const int kt1 = (int)min((int64_t)T, (int64_t)kt0 + (u_end - u));
  u += kt1 - kt0;
  const int b = (int)(rbg / a.row_blocks), rb = (int)(rbg % a.row_blocks);
  const int split = (int)blockIdx.x - attend_owner(rbg * T, U, G);
  const int row0 = rb * C::ROWS + wave * QB * 32;
  const int key_begin = kt0 * BN;
  const int key_end = min(a.n_valid, kt1 * BN);
  const int n_tiles = kt1 - kt0;
  __syncthreads();  // the previous segment's LDS tiles are no longer read

  // Bounds-checked views of this batch element's ring, ending at key_end.
  const int kend = key_end > 0 ? key_end : 0;
  const __amdgpu_buffer_rsrc_t rs_c = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.c_kv + (size_t)b * a.geo.ring_tokens * DC), (short)0, kend * DC * 2, kRawBufferWord3);
  const __amdgpu_buffer_rsrc_t rs_r = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.k_r + (size_t)b * a.geo.ring_tokens * DR), (short)0, kend * DR * 2, kRawBufferWord3);
  const u32x4 zero = {0, 0, 0, 0};


  // queries of this wave, B-operand layout: lane holds row l32, dims ks*16 + 8g .. +8
  bf16x8 q[QB][C::KSTEPS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = row0 + qb * 32 + l32;
    const uint16_t* src = a.qcat + ((size_t)b * rows_b + (r < rows_b ? r : 0)) * C::DQKP;
#pragma unroll
    for (int ks = 0; ks < C::KSTEPS; ++ks)
      q[qb][ks] = as_bf16x8(r < rows_b ? ldg16(src + ks * 16 + 8 * g) : zero);
  }

  f32x16 o[QB][C::DVB];
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = kNegInf;
    l_run[qb] = 0.f;
#pragma unroll
    for (int d = 0; d < C::DVB; ++d) o[qb][d] = f32x16{};
  }

  // Per-thread staging chunks: fixed (row, column) of the tile, so only the tile base moves.
  u32x4 pre_c[C::CPT_C], pre_r[C::CPT_R];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::CPT_C; ++i) {
      const int c = tid + i * C::NT;
      const uint32_t off = (uint32_t)((k0 + c / C::OCT_C) * DC + (c % C::OCT_C) * 8) * 2u;
      pre_c[i] = (C::CH_C % C::NT == 0 || c < C::CH_C)
                     ? __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs_c, off, 0, 0))
                     : zero;
    }
#pragma unroll
    for (int i = 0; i < C::CPT_R; ++i) {
      const int c = tid + i * C::NT;
      const uint32_t off = (uint32_t)((k0 + c / C::OCT_R) * DR + (c % C::OCT_R) * 8) * 2u;
      pre_r[i] = (C::CH_R % C::NT == 0 || c < C::CH_R)
                     ? __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs_r, off, 0, 0))
                     : zero;
    }
  };
  auto store_tile = [&](uint16_t* buf) {
#pragma unroll
    for (int i = 0; i < C::CPT_C; ++i) {
      const int c = tid + i * C::NT;
      if (C::CH_C % C::NT == 0 || c < C::CH_C)
        *reinterpret_cast<u32x4*>(&buf[(c / C::OCT_C) * C::STRIDE + (c % C::OCT_C) * 8]) = pre_c[i];
    }
#pragma unroll
    for (int i = 0; i < C::CPT_R; ++i) {
      const int c = tid + i * C::NT;
      if (C::CH_R % C::NT == 0 || c < C::CH_R)
        *reinterpret_cast<u32x4*>(&buf[(c / C::OCT_R) * C::STRIDE + DC + (c % C::OCT_R) * 8]) = pre_r[i];
    }
  };
  // S^T for one tile, both query blocks sharing each K operand read
  auto scores = [&](const uint16_t* buf, f32x16 (&s)[QB][C::KB]) {
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) s[qb][kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < C::KSTEPS; ++ks) {
        const bf16x8 k = as_bf16x8(
            *reinterpret_cast<const u32x4*>(&buf[(kb * 32 + l32) * C::STRIDE + ks * 16 + 8 * g]));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[qb][kb] = mfma32(k, q[qb][ks], s[qb][kb]);
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
      float m = kNegInf;
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) m = fmaxf(m, s[qb][kb][r]);
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
        for (int d = 0; d < C::DVB; ++d) {
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

  const int tr_row = (lane & 15) >> 2;
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // One pipelined step. s_cur holds tile t's scores, already masked, with m_run high enough
  // for them. Block A: scores of tile t+1 (MFMA) and tile t's exponentials (VALU). Block B: PV
  // of tile t (MFMA) and staging of tile t+2. After the barrier: masking and max of tile t+1.
  auto step = [&](int t, f32x16 (&s_cur)[QB][C::KB], f32x16 (&s_nxt)[QB][C::KB],
                  const uint16_t* cur, const uint16_t* nxt, uint16_t* stg) {
    const int kbase = key_begin + t * BN;

    // ---- block A: scores of tile t+1 and exponentials of tile t ----------------------------
    // The two waves sharing a SIMD (wave w and w + NW/2) take the two halves in opposite
    // order, so one's exponentials run while the other's score MFMAs do.
    load_tile(kbase + 2 * BN);
    bf16x8 pb[QB][2 * C::KB];
    // The row sum is taken over the bf16-rounded probabilities, the same values the PV MFMA
    // multiplies, so numerator and denominator see identical weights.
    auto exps = [&]() {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float acc = l_run[qb];
#pragma unroll
        for (int kb = 0; kb < C::KB; ++kb) {
          f32x16 p;
#pragma unroll
          for (int r = 0; r < 16; ++r) p[r] = fast_exp2(s_cur[qb][kb][r] - m_run[qb]);
          const f32x8 lo = {p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]};
          const f32x8 hi = {p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]};
          pb[qb][2 * kb] = to_bf16x8(lo);
          pb[qb][2 * kb + 1] = to_bf16x8(hi);
          acc = sum_bf16x8(pb[qb][2 * kb], acc);
          acc = sum_bf16x8(pb[qb][2 * kb + 1], acc);
        }
        l_run[qb] = acc;
      }
    };
    if (wave < NW / 2) {
      scores(nxt, s_nxt);
      exps();
    } else {
      exps();
      scores(nxt, s_nxt);
    }

    // ---- block B ---------------------------------------------------------------------------
    const lds_u16* vb = as_lds(cur) + (4 * g + tr_row) * C::STRIDE + tr_col;
#pragma unroll
    for (int kk = 0; kk < 2 * C::KB; ++kk) {
#pragma unroll
      for (int d = 0; d < C::DVB; ++d) {
        const i16x4 lo = lds_read_tr(vb + kk * 16 * C::STRIDE + d * 32);
        const i16x4 hi = lds_read_tr(vb + (kk * 16 + 8) * C::STRIDE + d * 32);
        const bf16x8 v = join_bf16x8(lo, hi);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) o[qb][d] = mfma32(v, pb[qb][kk], o[qb][d]);
      }
    }
    store_tile(stg);
    __syncthreads();
    if (kbase + 2 * BN > key_end) mask_tail(kbase + BN, s_nxt);  // only near the split's end
    own_max_of(s_nxt);
    raise_max_if_needed();
  };

  if (n_tiles > 0) {
    load_tile(key_begin);
    store_tile(tile[0]);
    load_tile(key_begin + BN);
    store_tile(tile[1]);
  }
  __syncthreads();

  f32x16 s_a[QB][C::KB], s_b[QB][C::KB];
  if (n_tiles > 0) {
    scores(tile[0], s_a);
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

  // ---- write unnormalized O_lat and (max, sum) of this split -------------------------------
  const size_t total_rows = (size_t)a.batch * rows_b;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l_tot = half_swap_sum(l_run[qb]);
    const int r = row0 + qb * 32 + l32;
    if (r >= rows_b) continue;
    const size_t grow_i = (size_t)b * rows_b + r;
    float* op = a.o_part + ((size_t)split * total_rows + grow_i) * DC;
#pragma unroll
    for (int d = 0; d < C::DVB; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = d * 32 + 8 * i + 4 * g;
        if (c < DC) {
          const f32x4 v = {o[qb][d][4 * i], o[qb][d][4 * i + 1], o[qb][d][4 * i + 2], o[qb][d][4 * i + 3]};
          *reinterpret_cast<f32x4*>(op + c) = v;
        }
      }
    if (g == 0) {
      float* ml = a.ml_part + ((size_t)split * total_rows + grow_i) * 2;
      ml[0] = m_run[qb];
      ml[1] = l_tot;
    }
  }
  }  // segments
}

// ---------------------------------------------------------------------------------------------
// out_proj: grid (ceil(Nq/128), H, B), 4 waves x 32 tokens, one head per workgroup.
// out^T[v][token] = W_UV_h[v][c] o_lat^T[c][token], where o_lat merges the key splits:
// o_lat = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
// ---------------------------------------------------------------------------------------------
template <int DC, int NVB>  // NVB = d_v / 32
__global__ __launch_bounds__(256) void out_proj_kernel(const AttendArgs a) {
  constexpr int KS = DC / 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int h = blockIdx.y, b = blockIdx.z;
  const int H = a.n_heads, dv = a.d_v, Nq = a.geo.chunk_tokens;
  const int n = blockIdx.x * 128 + wave * 32 + l32;
  const bool ok = n < Nq;
  const size_t total_rows = (size_t)a.batch * Nq * H;
  const size_t row = ((size_t)b * Nq + (ok ? n : 0)) * H + h;

  // partial results of this row's row block: one per workgroup that processed part of it
  const int64_t rbg = (int64_t)b * a.row_blocks + (int)((row - (size_t)b * Nq * H) / a.att_rows);
  const int n_seg = attend_owner(rbg * a.tiles_per_row + a.tiles_per_row - 1, a.units, a.n_wg) -
                    attend_owner(rbg * a.tiles_per_row, a.units, a.n_wg) + 1;
  float M = kNegInf;
  for (int s = 0; s < n_seg; ++s) M = fmaxf(M, a.ml_part[((size_t)s * total_rows + row) * 2]);
  float L = 0.f;
  for (int s = 0; s < n_seg; ++s) {
    const float* ml = a.ml_part + ((size_t)s * total_rows + row) * 2;
    L += fast_exp2(ml[0] - M) * ml[1];
  }
  const float invL = ok ? 1.f / L : 0.f;

  const uint16_t* w = a.w_uv + (size_t)h * dv * DC;
  f32x16 acc[NVB];
#pragma unroll
  for (int vb = 0; vb < NVB; ++vb) acc[vb] = f32x16{};

  for (int ks = 0; ks < KS; ++ks) {
    const int c0 = ks * 16 + 8 * g;
    f32x8 ov = {};
    for (int s = 0; s < n_seg; ++s) {
      const float coef = ok ? fast_exp2(a.ml_part[((size_t)s * total_rows + row) * 2] - M) * invL : 0.f;
      const f32x4* src = reinterpret_cast<const f32x4*>(a.o_part + ((size_t)s * total_rows + row) * DC + c0);
      const f32x4 v0 = src[0], v1 = src[1];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ov[e] += coef * v0[e];
        ov[4 + e] += coef * v1[e];
      }
    }
    const bf16x8 bo = to_bf16x8(ov);
#pragma unroll
    for (int vb = 0; vb < NVB; ++vb) {
      const bf16x8 aw = as_bf16x8(ldg16(w + (size_t)(vb * 32 + l32) * DC + c0));
      acc[vb] = mfma32(aw, bo, acc[vb]);
    }
  }
  if (!ok) return;
  uint16_t* dst = a.out + row * dv;
#pragma unroll
  for (int vb = 0; vb < NVB; ++vb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 v = {acc[vb][4 * i], acc[vb][4 * i + 1], acc[vb][4 * i + 2], acc[vb][4 * i + 3]};
      *reinterpret_cast<bf16x4*>(dst + vb * 32 + 8 * i + 4 * g) = to_bf16x4(v);
    }
  }
}

// Tile shapes per supported (d_c, d_rope).
template <int DC, int DR> struct AttShape;
template <> struct AttShape<192, 32> { static constexpr int QB = 1, NW = 8, BN = 32; };
template <> struct AttShape<16, 8> { static constexpr int QB = 1, NW = 4, BN = 32; };

template <int DC, int DR>
hipError_t launch_attend_t(const AttendArgs& a, hipStream_t s) {
  using S = AttShape<DC, DR>;
  using C = AttCfg<DC, DR, S::QB, S::NW, S::BN>;
  const dim3 grid(a.n_wg);
  hipLaunchKernelGGL((latent_attend_kernel<DC, DR, S::QB, S::NW, S::BN>), grid, dim3(C::NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace

bool latent_attend_supported(int d_c, int d_rope) {
  return (d_c == 192 && d_rope == 32) || (d_c == 16 && d_rope == 8);
}

int latent_attend_rows_per_block(int d_c, int d_rope) {
  if (d_c == 192 && d_rope == 32) return AttCfg<192, 32, AttShape<192, 32>::QB, AttShape<192, 32>::NW, AttShape<192, 32>::BN>::ROWS;
  return AttCfg<16, 8, AttShape<16, 8>::QB, AttShape<16, 8>::NW, AttShape<16, 8>::BN>::ROWS;
}

int latent_attend_keys_per_tile(int d_c, int d_rope) {
  if (d_c == 192 && d_rope == 32) return AttShape<192, 32>::BN;
  return AttShape<16, 8>::BN;
}

hipError_t launch_q_absorb(const AttendArgs& a, hipStream_t s) {
  const dim3 grid((a.geo.chunk_tokens + 127) / 128, a.n_heads, a.batch);
  if (a.d_c == 192 && a.d_rope == 32) {
    const size_t lds = (size_t)a.d_nope * (192 + 8) * 2;
    hipLaunchKernelGGL((q_absorb_kernel<192, 32>), grid, dim3(256), lds, s, a);
  } else if (a.d_c == 16 && a.d_rope == 8) {
    const size_t lds = (size_t)a.d_nope * (32 + 8) * 2;
    hipLaunchKernelGGL((q_absorb_kernel<16, 8>), grid, dim3(256), lds, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_latent_attend(const AttendArgs& a, hipStream_t s) {
  if (a.d_c == 192 && a.d_rope == 32) return launch_attend_t<192, 32>(a, s);
  if (a.d_c == 16 && a.d_rope == 8) return launch_attend_t<16, 8>(a, s);
  return hipErrorInvalidValue;
}

template <int DC>
hipError_t launch_out_proj_t(const AttendArgs& a, hipStream_t s) {
  const dim3 grid((a.geo.chunk_tokens + 127) / 128, a.n_heads, a.batch);
  switch (a.d_v / 32) {
    case 1: hipLaunchKernelGGL((out_proj_kernel<DC, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((out_proj_kernel<DC, 2>), grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((out_proj_kernel<DC, 3>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((out_proj_kernel<DC, 4>), grid, dim3(256), 0, s, a); break;
    case 5: hipLaunchKernelGGL((out_proj_kernel<DC, 5>), grid, dim3(256), 0, s, a); break;
    case 6: hipLaunchKernelGGL((out_proj_kernel<DC, 6>), grid, dim3(256), 0, s, a); break;
    case 7: hipLaunchKernelGGL((out_proj_kernel<DC, 7>), grid, dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL((out_proj_kernel<DC, 8>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_out_proj(const AttendArgs& a, hipStream_t s) {
  if (a.d_c == 192) return launch_out_proj_t<192>(a, s);
  if (a.d_c == 16) return launch_out_proj_t<16>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace vmla
