// The whole attention layer in latent form (App. "Inference-Time Reparameterization", Eqs. 8-11):
//
//   prepare_weights   once per model load: W_down^Q padded to whole 64-column chunks; per head
//                     [A_h^T diag(g_Q) ; W_R,h^Q diag(g_Q)] with A_h = (W_up,h^Q)^T W_up,h^K (the
//                     RMSNorm gain g_Q of c^Q folded into the columns); B_h = W_h^O W_up,h^V
//   gemm (store)      u = W_down^Q x, bf16 (c^Q before its RMSNorm)
//   gemm (q_cat)      q_cat row (token, head) = [A_h^T c^Q, RoPE(W_R,h^Q c^Q)] * scale * log2 e,
//                     with c^Q = g_Q u / rms(u): 1 / rms(u) is a per-token factor, taken from the
//                     sum of squares of u that the kernel accumulates from its own operand reads
//   latent_attend     unchanged
//   latent_merge      o_lat = exact merge of the key splits, bf16 [token][H d_c] (+ zero padding)
//   gemm (store)      y = sum_h B_h o_lat_h = [B_1 .. B_H] o_lat
//
// gemm: out^T[o][token] = A[o][:] . B[token][:], A = weight rows [N][K], B = token rows [M][K],
// both row-major with K % 64 == 0. A workgroup of 8 waves (two per SIMD) takes 128 tokens and
// 128 or 256 outputs, each wave 32 tokens x 64 or 128 outputs with MFMA 32x32x16; the
// contraction streams through LDS stages of 64 columns filled by direct global-to-LDS loads
// (chunk index XOR (row / 2) mod 8). Tiles are numbered token-block-major and dealt to the XCDs
// in contiguous ranges. Rows past M or N are clamped to the last row and their results discarded.
#include "vmla_device.h"

namespace vmla {
namespace {

__device__ __forceinline__ int gm_swz(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }
constexpr int kGmKC = 64;  // contraction columns per LDS stage

// Tile shape: TT token rows x TO outputs per workgroup, WT x WO waves (each 32 tokens x TO / WO
// outputs), ST stages of 64 columns, at least MINB workgroups resident per CU. XCD: tiles are
// numbered token-block-major and each XCD takes a contiguous range of them (workgroup w runs on
// XCD w mod 8), so that the workgroups sharing a token block share that XCD's L2.
template <int TT, int TO, int WT, int WO, int ST, int MINB, bool XCD = false>
struct GemmShape {
  static constexpr int kTok = TT, kOut = TO, kWT = WT, kWO = WO, kStages = ST, kMinBlocks = MINB;
  static constexpr bool kXcdMap = XCD;
  static constexpr int kWaves = WT * WO, kThreads = 64 * kWaves;
  static constexpr int kRows = TT + TO;              // LDS rows per stage (tokens, then outputs)
  static constexpr int kLoadsPerWave = kRows * 8 / 64 / kWaves;  // 1 KB loads per wave per stage
  static constexpr int kMO = TO / WO / 32;           // 32x32 output blocks per wave
  static_assert(TT == 32 * WT && TO % (32 * WO) == 0, "wave tiling");
  static_assert(kRows * 8 % (64 * kWaves) == 0, "stage loads split evenly over the waves");
  static constexpr size_t kLdsBytes = (size_t)ST * kRows * kGmKC * 2;
};

template <int EPI, class P>
__global__ __launch_bounds__(P::kThreads, P::kMinBlocks) void gemm_nt_kernel(const GemmArgs a) {
  constexpr int TT = P::kTok, TO = P::kOut, ST = P::kStages, NW = P::kWaves, MO = P::kMO;
  constexpr int LPW = P::kLoadsPerWave, WOUT = 32 * MO;
  __shared__ __attribute__((aligned(16))) uint16_t stage[ST][P::kRows * kGmKC];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wt = wave % P::kWT, wo = wave / P::kWT;
  const int g = lane >> 5, l32 = lane & 31;
  int tx = blockIdx.x, ty = blockIdx.y;
  if constexpr (P::kXcdMap) {
    const int nty = (a.N + TO - 1) / TO, G = gridDim.x, id = blockIdx.x;
    const int xcd = id & 7, L = xcd * (G >> 3) + min(xcd, G & 7) + (id >> 3);
    tx = L / nty;
    ty = L % nty;
  }
  const int n0 = tx * TT, o0 = ty * TO;
  const int K = a.K;

  const uint16_t* src[LPW];
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    const int p = (wave + NW * i) * 64 + lane;
    const int r = p >> 3, cs = p & 7;
    const int c = cs ^ ((r >> 1) & 7);
    const uint16_t* row = r < TT ? a.b + (size_t)min(n0 + r, a.M - 1) * K
                                 : a.a + (size_t)min(o0 + r - TT, a.N - 1) * K;
    src[i] = row + c * 8;
  }
  auto issue = [&](int chunk) {
    uint16_t* st = stage[chunk % ST];
#pragma unroll
    for (int i = 0; i < LPW; ++i)
      lds_dma16(src[i] + chunk * kGmKC,
                __builtin_amdgcn_readfirstlane(lds_addr(st + (wave + NW * i) * 512)));
  };

  f32x16 acc[MO];
#pragma unroll
  for (int m = 0; m < MO; ++m) acc[m] = f32x16{};
  float ssq = 0.f;  // q_cat epilogue: this lane's half of the token row's sum of squares
  const int nchunks = K / kGmKC;
#pragma unroll
  for (int c = 0; c < ST - 1; ++c)
    if (c < nchunks) issue(c);
  for (int i = 0; i < nchunks; ++i) {
    if (i + ST - 2 < nchunks) wait_vmcnt<(ST - 2) * LPW>();
    else wait_vmcnt<0>();
    __syncthreads();  // chunk i is in LDS for every wave; chunk i-1 is no longer read
    if (i + ST - 1 < nchunks) issue(i + ST - 1);
    const uint16_t* st = stage[i % ST];
#pragma unroll
    for (int ks = 0; ks < kGmKC / 16; ++ks) {
      const int c = ks * 2 + g;
      const bf16x8 bx =
          as_bf16x8(*reinterpret_cast<const u32x4*>(&st[gm_swz(wt * 32 + l32, c) * 8]));
      if constexpr (EPI == kEpiQcat) {  // widen each bf16 by its bit pattern, square in fp32
        const u32x4 w = as_u32x4(bx);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(w[e] << 16), hi = __uint_as_float(w[e] & 0xffff0000u);
          ssq = fmaf(lo, lo, ssq);
          ssq = fmaf(hi, hi, ssq);
        }
      }
#pragma unroll
      for (int m = 0; m < MO; ++m) {
        const bf16x8 aw = as_bf16x8(*reinterpret_cast<const u32x4*>(
            &st[gm_swz(TT + wo * WOUT + m * 32 + l32, c) * 8]));
        acc[m] = mfma32(aw, bx, acc[m]);
      }
    }
  }

  // epilogue: lane holds token n0 + 32 wt + l32 and outputs o0 + wo WOUT + 32 m + 8 i + 4 g + j
  const int ob = o0 + wo * WOUT;
  if constexpr (EPI == kEpiHeads) {
    // through LDS, so that every store is a whole 16-byte chunk of 8 consecutive outputs of one
    // token (head_w % 8 == 0 keeps a chunk inside one head): each wave's 32 token rows x WOUT
    // outputs go to its own LDS tile, then its lanes copy them out row by row
    constexpr int OTS = WOUT + 8;  // tile row stride (elements)
    static_assert(NW * 32 * OTS <= ST * P::kRows * kGmKC, "output tiles fit the stage buffers");
    __syncthreads();               // every wave is done reading the stage buffers
    uint16_t* ot = &stage[0][0] + wave * 32 * OTS;
#pragma unroll
    for (int m = 0; m < MO; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 fv = {acc[m][4 * i], acc[m][4 * i + 1], acc[m][4 * i + 2], acc[m][4 * i + 3]};
        *reinterpret_cast<bf16x4*>(&ot[l32 * OTS + m * 32 + 8 * i + 4 * g]) = to_bf16x4(fv);
      }
    __syncthreads();  // the tile rows are read by other lanes than the ones that wrote them
#pragma unroll 4
    for (int it = lane; it < 32 * (WOUT / 8); it += 64) {
      const int tr = it / (WOUT / 8), ch = it % (WOUT / 8);
      const int tok = n0 + wt * 32 + tr, o = ob + ch * 8;
      if (tok < a.M && o < a.N)
        stg16(a.out + (size_t)tok * a.ldo + (size_t)(o / a.head_w) * a.head_ld + a.col_off +
                  o % a.head_w,
              *reinterpret_cast<const u32x4*>(&ot[tr * OTS + ch * 8]));
    }
    return;
  }
  const int t = n0 + wt * 32 + l32;
  float scale = 1.f;
  TokenPos pos{};
  if constexpr (EPI == kEpiQcat) {
    ssq = half_swap_sum(ssq);
    scale = a.qscale * rsqrtf(ssq / (float)a.q_norm_dim + a.eps);
    if (t < a.M) pos = rope_pos(a.geo, query_pos(a.geo, t % a.geo.q_count));
  }
  if (t >= a.M) return;
#pragma unroll
  for (int m = 0; m < MO; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = ob + m * 32 + 8 * i + 4 * g;
      if (o >= a.N) continue;
      float v[4] = {acc[m][4 * i], acc[m][4 * i + 1], acc[m][4 * i + 2], acc[m][4 * i + 3]};
      uint16_t* dst;
      if constexpr (EPI == kEpiQcat) {
        const int dqk = a.q_dc + a.q_dr;
        const int h = o / dqk, c = o % dqk;
        if (c >= a.q_dc) {  // channels c .. c+3 of the RoPE query: pairs (c - d_c)/2 and +1
          rope_rotate(a.rope, (c - a.q_dc) / 2, pos, v[0], v[1]);
          rope_rotate(a.rope, (c - a.q_dc) / 2 + 1, pos, v[2], v[3]);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] *= scale;
        dst = a.out + ((size_t)t * a.q_heads + h) * a.ldo + c;
      } else {
        dst = a.out + (size_t)t * a.ldo + o;
      }
      const f32x4 fv = {v[0], v[1], v[2], v[3]};
      *reinterpret_cast<bf16x4*>(dst) = to_bf16x4(fv);
    }
  if constexpr (EPI == kEpiQcat) {  // zero padding of each head's q_cat row
    const int dqk = a.q_dc + a.q_dr;
    if (ty == 0 && wo == 0 && g == 0)
      for (int h = 0; h < a.q_heads; ++h)
        for (int c = dqk; c < a.ldo; ++c) a.out[((size_t)t * a.q_heads + h) * a.ldo + c] = 0;
  }
}

// ---------------------------------------------------------------------------------------------
// latent_merge: one thread per (query row, 8 latent columns); query rows (token, head) in
// head-minor order. o_lat = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s, rounded to bf16 and
// stored at o_lat[token][h d_c + c] (row stride ld_olat); the threads past the rows zero the
// padding columns H d_c .. ld_olat of every token.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void latent_merge_kernel(const AttendArgs a, uint16_t* o_lat,
                                                           int ld_olat) {
  // 32-bit index arithmetic: the launcher keeps the thread count below 2^32
  const int DC = a.d_c, H = a.n_heads;
  const uint32_t gpr = (uint32_t)DC / 8;
  const int Nq = a.geo.q_count;
  const uint32_t rows_b = (uint32_t)(Nq * H);
  const uint32_t n_rows = (uint32_t)a.batch * rows_b;
  const uint32_t e = blockIdx.x * 256u + threadIdx.x;
  if (e >= n_rows * gpr) {
    const uint32_t pad_groups = (uint32_t)(ld_olat - H * DC) / 8;
    const uint32_t z = e - n_rows * gpr;
    if (pad_groups == 0 || z >= (uint32_t)a.batch * Nq * pad_groups) return;
    const int64_t tok = z / pad_groups;
    const int grp = (int)(z % pad_groups);
    *reinterpret_cast<u32x4*>(o_lat + tok * ld_olat + H * DC + grp * 8) = u32x4{0, 0, 0, 0};
    return;
  }
  const uint32_t R = e / gpr;  // global query row = token * H + h
  const int grp = (int)(e % gpr);
  const int b = (int)(R / rows_b), r = (int)(R % rows_b);
  const size_t total_rows = (size_t)n_rows;
  const int64_t rbg = (int64_t)b * a.row_blocks + r / a.att_rows;
  const int ns = attend_split_count(a, rbg);
  // the splits' loads are issued in groups (eight maxima, then four partial rows at a time), so
  // that rows split over many workgroups do not wait on one load per split; the sums still run
  // in split order
  float M = -__builtin_huge_valf();
  for (int s0 = 0; s0 < ns; s0 += 8) {
    float m[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      m[j] = s0 + j < ns ? a.ml_part[((size_t)(s0 + j) * total_rows + R) * 2] : -__builtin_huge_valf();
#pragma unroll
    for (int j = 0; j < 8; ++j) M = fmaxf(M, m[j]);
  }
  float L = 0.f;
  f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < ns; s0 += 4) {
    f32x2 ml[4];
    f32x4 vlo[4], vhi[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (s0 + j < ns) {
        const size_t base = (size_t)(s0 + j) * total_rows + R;
        ml[j] = *reinterpret_cast<const f32x2*>(a.ml_part + base * 2);
        const f32x4* src = reinterpret_cast<const f32x4*>(a.o_part + base * DC + grp * 8);
        vlo[j] = src[0];
        vhi[j] = src[1];
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (s0 + j < ns) {
        const float coef = fast_exp2(ml[j][0] - M);
        L += coef * ml[j][1];
        lo += coef * vlo[j];
        hi += coef * vhi[j];
      }
    }
  }
  const float il = 1.f / L;
  const f32x8 v = {lo[0] * il, lo[1] * il, lo[2] * il, lo[3] * il,
                   hi[0] * il, hi[1] * il, hi[2] * il, hi[3] * il};
  const int64_t tok = R / (uint32_t)H;
  const int h = (int)(R % (uint32_t)H);
  *reinterpret_cast<bf16x8*>(o_lat + tok * ld_olat + h * DC + grp * 8) = to_bf16x8(v);
}

// ---------------------------------------------------------------------------------------------
// prepare_weights: one thread per output element of the packed weights, fp32 sums, bf16 RNE.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void prepare_weights_kernel(const PrepArgs a) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int H = a.n_heads, DC = a.d_c, DR = a.d_rope, DN = a.d_nope, DV = a.d_v;
  const int dqk = DC + DR;
  const int64_t n1 = (int64_t)a.d_q_pad * a.d_model;
  const int64_t n2 = (int64_t)H * dqk * a.d_q_pad;
  const int64_t n3 = (int64_t)a.d_model * a.k_out_pad;
  float v = 0.f;
  uint16_t* dst;
  if (e < n1) {  // W_down^Q with zero rows past d_q
    const int r = (int)(e / a.d_model), k = (int)(e % a.d_model);
    dst = a.w_dq_pad + e;
    if (r < a.d_q) {
      *dst = a.w_dq[(size_t)r * a.d_model + k];
      return;
    }
  } else if (e < n1 + n2) {  // per head [A_h^T diag(g) ; W_R,h^Q diag(g)], zero columns past d_q
    const int64_t f = e - n1;
    const int row = (int)(f / a.d_q_pad), k = (int)(f % a.d_q_pad);
    const int h = row / dqk, c = row % dqk;
    dst = a.wq_cat + f;
    if (k < a.d_q) {
      const float gk = a.gamma_q ? bf16_bits_to_f32(a.gamma_q[k]) : 1.f;
      if (c < DC) {
        for (int n = 0; n < DN; ++n)
          v += bf16_bits_to_f32(a.w_uq[(size_t)(h * DN + n) * a.d_q + k]) *
               bf16_bits_to_f32(a.w_uk[(size_t)(h * DN + n) * DC + c]);
      } else {
        v = bf16_bits_to_f32(a.w_qr[(size_t)(h * DR + c - DC) * a.d_q + k]);
      }
      v *= gk;
    }
  } else if (e < n1 + n2 + n3) {  // B = [B_1 .. B_H], B_h = W_h^O W_up,h^V, zero columns past H d_c
    const int64_t f = e - n1 - n2;
    const int i = (int)(f / a.k_out_pad), j = (int)(f % a.k_out_pad);
    dst = a.b_o + f;
    if (j < H * DC) {
      const int h = j / DC, c = j % DC;
      for (int q = 0; q < DV; ++q)
        v += bf16_bits_to_f32(a.w_o[(size_t)i * H * DV + h * DV + q]) *
             bf16_bits_to_f32(a.w_uv[(size_t)(h * DV + q) * DC + c]);
    }
  } else {
    return;
  }
  *dst = to_bf16_bits(v);
}

}  // namespace

template <class P>
hipError_t launch_gemm_shape(const GemmArgs& a, hipStream_t s) {
  const int ntx = (a.M + P::kTok - 1) / P::kTok, nty = (a.N + P::kOut - 1) / P::kOut;
  const dim3 grid = P::kXcdMap ? dim3(ntx * nty) : dim3(ntx, nty);
  if (a.epi == kEpiQcat)
    hipLaunchKernelGGL((gemm_nt_kernel<kEpiQcat, P>), grid, dim3(P::kThreads), 0, s, a);
  else if (a.epi == kEpiHeads)
    hipLaunchKernelGGL((gemm_nt_kernel<kEpiHeads, P>), grid, dim3(P::kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((gemm_nt_kernel<kEpiStore, P>), grid, dim3(P::kThreads), 0, s, a);
  return hipGetLastError();
}

// Wide tiles (128 tokens x 256 outputs) carry twice the MFMA work per byte a CU takes in, and
// win once they fill most of the chip (Wan shape: q_up 58 -> 45 us, out_mix 57 -> 46 us); below
// that the 128 x 128 tiles keep every CU busy (q_down, 111 wide tiles: 21 -> 20 us).
using GemmWide = GemmShape<128, 256, 4, 2, 3, 1, true>;
using GemmSquare = GemmShape<128, 128, 4, 2, 4, 1, true>;

hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s) {
  // validated by the caller: K % 64 == 0, N % 4 == 0, M >= 1, N >= 1
  const int64_t wide_tiles = (int64_t)((a.M + GemmWide::kTok - 1) / GemmWide::kTok) *
                             ((a.N + GemmWide::kOut - 1) / GemmWide::kOut);
  if (wide_tiles >= 192) return launch_gemm_shape<GemmWide>(a, s);
  return launch_gemm_shape<GemmSquare>(a, s);
}

hipError_t launch_latent_merge(const AttendArgs& a, uint16_t* o_lat, int ld_olat, hipStream_t s) {
  const int64_t rows = (int64_t)a.batch * a.geo.q_count * a.n_heads;
  const int64_t pad = (int64_t)a.batch * a.geo.q_count * ((ld_olat - a.n_heads * a.d_c) / 8);
  const int64_t threads = rows * (a.d_c / 8) + pad;
  if (threads >= (int64_t(1) << 32) - 256) return hipErrorInvalidValue;  // 32-bit indices
  hipLaunchKernelGGL(latent_merge_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                     a, o_lat, ld_olat);
  return hipGetLastError();
}

hipError_t launch_prepare_weights(const PrepArgs& a, hipStream_t s) {
  const int64_t n = (int64_t)a.d_q_pad * a.d_model +
                    (int64_t)a.n_heads * (a.d_c + a.d_rope) * a.d_q_pad +
                    (int64_t)a.d_model * a.k_out_pad;
  hipLaunchKernelGGL(prepare_weights_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace vmla
