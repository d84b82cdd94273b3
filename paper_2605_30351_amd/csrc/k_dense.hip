// Dense per-head comparator: the KV cache that VideoMLA's latent cache replaces. Every token
// caches, per head h, K_h = W_K,h x rotated by 3D RoPE over the whole head and V_h = W_V,h x
// (the per-head keys and values of Eq. 2 without a shared latent); queries attend with standard
// softmax attention over the same sliding window (App. "Chunk-Causal Sliding-Window
// Attention"). Built here only to compare speed and memory with the latent path.
//
//   dense_cache_write  [K | V] = x [W_K; W_V]^T, a 128-token x 128-output MFMA tile per
//                      workgroup with LDS-staged operands; the K half is rotated and every
//                      head's [K_h | V_h] row is stored at the token's ring slot
//   dense_q_prep       q_cat[b][h][n] = RoPE_head(q[b][n][h]) * scale * log2(e), each head's
//                      rows padded with zeros to whole row blocks
//   (the attention itself is latent_attend_kernel with the dense tile layout)
//   dense_merge        merges the key splits exactly and writes out[b][n][h]
#include "vmla_device.h"

namespace vmla {
namespace {

constexpr float kNegInfD = -__builtin_huge_valf();

// ---------------------------------------------------------------------------------------------
// dense_cache_write: grid (ceil(Nq/128), 2 H d_head / 128, B), 4 waves; wave w computes the
// 128 outputs of the tile for tokens 32 w .. 32 w + 31 of the tile, out^T[o][token] with
// MFMA 32x32x16 (A = weight rows, B = token rows). The contraction over d_model streams
// through three LDS stages of 64 columns (x rows then weight rows, 8 chunks of 16 bytes per
// row, chunk index XOR ((row / 2) mod 8) so that 16-row operand reads are conflict-free),
// filled two stages ahead by direct global-to-LDS loads.
// ---------------------------------------------------------------------------------------------
constexpr int kDwTok = 128, kDwOut = 128, kDwKC = 64, kDwStages = 3;
constexpr int kDwRows = kDwTok + kDwOut;          // staged rows per stage
constexpr int kDwLoads = kDwRows * 8 / 64;        // 1 KB loads per stage (32)
constexpr int kDwMaxPairs = 64;  // RoPE pairs whose angle table fits the stage memory

__device__ __forceinline__ int dw_swz(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

__global__ __launch_bounds__(256, 1) void dense_cache_write_kernel(const DenseWriteArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t stage[kDwStages][kDwRows * kDwKC];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, l32 = lane & 31;
  const int b = blockIdx.z;
  const int n0 = blockIdx.x * kDwTok, o0 = blockIdx.y * kDwOut;
  const int dm = a.d_model, H = a.n_heads, DH = a.d_head;
  const int n_tok = a.geo.chunk_tokens;
  const int hd = H * DH;  // outputs of one of K, V

  // this wave's loads j = wave + 4 i: chunk slots 64 j .. 64 j + 63 of a stage
  const uint16_t* src[kDwLoads / 4];
#pragma unroll
  for (int i = 0; i < kDwLoads / 4; ++i) {
    const int p = (wave + 4 * i) * 64 + lane;
    const int r = p >> 3, cs = p & 7;
    const int c = cs ^ ((r >> 1) & 7);
    const uint16_t* row;
    if (r < kDwTok) {
      const int n = min(n0 + r, n_tok - 1);
      row = a.x + ((size_t)b * n_tok + n) * dm;
    } else {
      const int o = o0 + r - kDwTok;
      row = o < hd ? a.w_k + (size_t)o * dm : a.w_v + (size_t)(o - hd) * dm;
    }
    src[i] = row + c * 8;
  }
  auto issue = [&](int chunk) {
    uint16_t* st = stage[chunk % kDwStages];
#pragma unroll
    for (int i = 0; i < kDwLoads / 4; ++i)
      lds_dma16(src[i] + chunk * kDwKC,
                __builtin_amdgcn_readfirstlane(lds_addr(st + (wave + 4 * i) * 512)));
  };

  f32x16 acc[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) acc[m] = f32x16{};
  const int nchunks = dm / kDwKC;
#pragma unroll
  for (int c = 0; c < kDwStages - 1; ++c)
    if (c < nchunks) issue(c);
  for (int i = 0; i < nchunks; ++i) {
    if (i + kDwStages - 2 < nchunks) wait_vmcnt<(kDwStages - 2) * (kDwLoads / 4)>();
    else wait_vmcnt<0>();
    __syncthreads();  // chunk i is in LDS for every wave; chunk i-1 is no longer read
    if (i + kDwStages - 1 < nchunks) issue(i + kDwStages - 1);
    const uint16_t* st = stage[i % kDwStages];
#pragma unroll
    for (int ks = 0; ks < kDwKC / 16; ++ks) {
      const int c = ks * 2 + g;
      const bf16x8 bx =
          as_bf16x8(*reinterpret_cast<const u32x4*>(&st[dw_swz(wave * 32 + l32, c) * 8]));
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const bf16x8 aw = as_bf16x8(
            *reinterpret_cast<const u32x4*>(&st[dw_swz(kDwTok + m * 32 + l32, c) * 8]));
        acc[m] = mfma32(aw, bx, acc[m]);
      }
    }
  }

  // (cos, sin) of every (token, RoPE pair) of a tile holding K outputs, computed once into the
  // free stage memory: wave w takes the pairs w, w + 4, .. (a pair index uniform across the wave,
  // so that its table entries are read by scalar loads), lanes the tile's tokens. Rows are padded
  // by one entry so that the epilogue's reads (32 tokens at one pair) hit distinct banks. Heads
  // wider than 2 kDwMaxPairs take the angles per lane instead.
  const int npair = DH / 2, cs_ld = npair + 1;
  const bool cs_table = o0 < hd && npair <= kDwMaxPairs;  // uniform
  const f32x2* cs_tab = reinterpret_cast<const f32x2*>(&stage[0][0]);
  if (cs_table) {
    f32x2* tab = reinterpret_cast<f32x2*>(&stage[0][0]);
    __syncthreads();  // every wave is past its last stage read
    TokenPos tp[kDwTok / 64];
#pragma unroll
    for (int k = 0; k < kDwTok / 64; ++k) tp[k] = token_pos(a.geo, min(n0 + lane + 64 * k, n_tok - 1));
    for (int p = wave; p < npair; p += 4) {
      const RopePair rp = rope_pair(a.rope, __builtin_amdgcn_readfirstlane(p));
#pragma unroll
      for (int k = 0; k < kDwTok / 64; ++k) tab[(lane + 64 * k) * cs_ld + p] = rope_cos_sin(rp, tp[k]);
    }
    __syncthreads();
  }

  // epilogue: lane holds token n, outputs o0 + 32 m + 8 i + 4 g + j (4 consecutive channels of
  // one head: two RoPE pairs when they belong to K)
  const int n = n0 + wave * 32 + l32;
  if (n >= n_tok) return;
  const TokenPos pos = token_pos(a.geo, n);
  const int64_t slot = ring_slot(a.geo, pos);
  uint16_t* dst = a.kv + ((size_t)b * a.geo.ring_tokens + slot) * H * 2 * DH;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = o0 + m * 32 + 8 * i + 4 * g;
      float v[4] = {acc[m][4 * i], acc[m][4 * i + 1], acc[m][4 * i + 2], acc[m][4 * i + 3]};
      const bool is_k = o < hd;
      const int oo = is_k ? o : o - hd;
      const int h = oo / DH, ch = oo % DH;
      if (is_k && cs_table) {
        const f32x2* row = cs_tab + (wave * 32 + l32) * cs_ld + ch / 2;
        rotate_by(row[0], v[0], v[1]);
        rotate_by(row[1], v[2], v[3]);
      } else if (is_k) {
        rope_rotate(a.rope, ch / 2, pos, v[0], v[1]);
        rope_rotate(a.rope, ch / 2 + 1, pos, v[2], v[3]);
      }
      const f32x4 fv = {v[0], v[1], v[2], v[3]};
      *reinterpret_cast<bf16x4*>(dst + (size_t)h * 2 * DH + (is_k ? 0 : DH) + ch) = to_bf16x4(fv);
    }
  if (a.slots && b == 0 && blockIdx.y == 0 && g == 0) a.slots[n] = (int32_t)slot;
}

// ---------------------------------------------------------------------------------------------
// dense_q_prep: grid (nq_pad / 4, B), 256 threads = 4 tokens x 64 RoPE pairs; each thread takes
// the angle of its (token, pair) once and applies it to that pair of every head.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void dense_q_prep_kernel(const AttendArgs a) {
  const int t = threadIdx.x >> 6, p = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + t, b = blockIdx.y;
  const int H = a.n_heads, DH = a.d_v, Nq = a.geo.q_count;
  if (2 * p >= DH) return;
  float cs = 1.f, sn = 0.f;
  if (n < Nq) rope_rotate(a.rope, p, query_pos(a.geo, n), cs, sn);  // (1, 0) -> (cos, sin)
  for (int h = 0; h < H; ++h) {
    uint32_t packed = 0;
    if (n < Nq) {
      const uint32_t raw =
          *reinterpret_cast<const uint32_t*>(a.q + (((size_t)b * Nq + n) * H + h) * DH + 2 * p);
      const float u = bf16_bits_to_f32((uint16_t)(raw & 0xffff));
      const float v = bf16_bits_to_f32((uint16_t)(raw >> 16));
      packed = (uint32_t)to_bf16_bits((u * cs - v * sn) * a.qscale) |
               ((uint32_t)to_bf16_bits((u * sn + v * cs) * a.qscale) << 16);
    }
    *reinterpret_cast<uint32_t*>(a.qcat + (((size_t)b * H + h) * a.nq_pad + n) * DH + 2 * p) = packed;
  }
}

// ---------------------------------------------------------------------------------------------
// mat_q_prep (materialized-K/V path): per-head query rows [q_nope ; RoPE_3D(q_R)] * scale *
// log2 e (Eq. 4 and Eq. 6, the training form), d_nope + d_rope wide, head-major and padded like
// dense_q_prep's. Grid (nq_pad / 4, B), 256 threads = 4 tokens x 64 lanes over the row's channel
// pairs; a RoPE pair takes its angle once and applies it to every head.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void mat_q_prep_kernel(const AttendArgs a) {
  const int t = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + t, b = blockIdx.y;
  const int H = a.n_heads, DN = a.d_nope, DR = a.d_rope, DH = a.dqk_pad, Nq = a.geo.q_count;
  for (int p = lane; 2 * p < DH; p += 64) {  // channel pair p of the d_nope + d_rope wide row
    const bool rope = 2 * p >= DN;
    const int pr = p - DN / 2;  // RoPE pair (when rope)
    float cs = 1.f, sn = 0.f;
    if (rope && n < Nq) rope_rotate(a.rope, pr, query_pos(a.geo, n), cs, sn);  // (1,0) -> (cos, sin)
    for (int h = 0; h < H; ++h) {
      uint32_t packed = 0;
      if (n < Nq) {
        const size_t row = ((size_t)b * Nq + n) * H + h;
        const uint32_t raw = rope ? *reinterpret_cast<const uint32_t*>(a.q_r + row * DR + 2 * pr)
                                  : *reinterpret_cast<const uint32_t*>(a.q_nope + row * DN + 2 * p);
        const float u = bf16_bits_to_f32((uint16_t)(raw & 0xffff));
        const float v = bf16_bits_to_f32((uint16_t)(raw >> 16));
        packed = (uint32_t)to_bf16_bits((u * cs - v * sn) * a.qscale) |
                 ((uint32_t)to_bf16_bits((u * sn + v * cs) * a.qscale) << 16);
      }
      *reinterpret_cast<uint32_t*>(a.qcat + (((size_t)b * H + h) * a.nq_pad + n) * DH + 2 * p) = packed;
    }
  }
}

// mat_rope_fill: the head-shared RoPE key of every valid slot (rotated at write) copied into
// channels d_nope .. d_nope + d_rope of every head's K_h row of the materialized ring
// [B][ring][H][d_nope + d_rope + d_v]. One thread per (batch, slot, head, 16-byte chunk).
__global__ __launch_bounds__(256) void mat_rope_fill_kernel(const AttendArgs a, uint16_t* kv) {
  const int H = a.n_heads, DR = a.d_rope, cpk = DR / 8, LD = a.dqk_pad + a.d_v;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_b = (int64_t)a.n_valid * H * cpk;
  if (e >= per_b * a.batch) return;
  const int b = (int)(e / per_b);
  const int64_t r = e - b * per_b;
  const int ch = (int)(r % cpk);
  const int64_t jh = r / cpk;
  const int h = (int)(jh % H);
  const int64_t j = jh / H;
  const size_t slot = (size_t)b * a.geo.ring_tokens + j;
  stg16(kv + (slot * H + h) * LD + a.d_nope + ch * 8, ldg16(a.k_r + slot * DR + ch * 8));
}

// ---------------------------------------------------------------------------------------------
// dense_merge: one thread per (output row, 8 columns), in the partial results' head-major row
// order [B][H][Nq], so that a wave reads consecutive partial rows; output rows are stored in
// [B][Nq][H] order.
// out = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s over the key splits s of the row.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void dense_merge_kernel(const AttendArgs a) {
  // 32-bit index arithmetic: the launcher keeps the thread count below 2^32
  const int DH = a.d_v;
  const uint32_t gpr = (uint32_t)DH / 8;
  const uint32_t e = blockIdx.x * 256u + threadIdx.x;
  const uint32_t H = (uint32_t)a.n_heads, Nq = (uint32_t)a.geo.q_count;
  const uint32_t n_out = (uint32_t)a.batch * Nq * H;
  const uint32_t Rp = e / gpr;  // row in [B][H][Nq] order
  const int grp = (int)(e % gpr);
  if (Rp >= n_out) return;
  const int n = (int)(Rp % Nq);
  const uint32_t bh = Rp / Nq;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t R = ((int64_t)b * Nq + n) * H + h;  // output row
  const int rows_b = H * a.nq_pad;
  const int r = h * a.nq_pad + n;                    // row within the batch element
  const size_t total_rows = (size_t)a.batch * rows_b;
  const size_t orow = (size_t)b * rows_b + r;
  const int64_t rbg = (int64_t)b * a.row_blocks + r / a.att_rows;
  const int ns = attend_split_count(a, rbg);
  float M = kNegInfD;
  float L = 0.f;
  f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
  if (ns <= 4) {
    // every load of the row's splits issued together (one memory round trip), summed in split
    // order as below
    f32x2 ml[4];
    f32x4 vlo[4], vhi[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s < ns) {
        const size_t base = (size_t)s * total_rows + orow;
        ml[s] = *reinterpret_cast<const f32x2*>(a.ml_part + base * 2);
        const f32x4* src = reinterpret_cast<const f32x4*>(a.o_part + base * DH + grp * 8);
        vlo[s] = src[0];
        vhi[s] = src[1];
      }
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
      if (s < ns) M = fmaxf(M, ml[s][0]);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s < ns) {
        const float coef = fast_exp2(ml[s][0] - M);
        L += coef * ml[s][1];
        lo += coef * vlo[s];
        hi += coef * vhi[s];
      }
    }
  } else {
    for (int s = 0; s < ns; ++s) M = fmaxf(M, a.ml_part[((size_t)s * total_rows + orow) * 2]);
    for (int s = 0; s < ns; ++s) {
      const float* ml = a.ml_part + ((size_t)s * total_rows + orow) * 2;
      const float coef = fast_exp2(ml[0] - M);
      L += coef * ml[1];
      const f32x4* src = reinterpret_cast<const f32x4*>(a.o_part + ((size_t)s * total_rows + orow) * DH + grp * 8);
      lo += coef * src[0];
      hi += coef * src[1];
    }
  }
  const float il = 1.f / L;
  const f32x8 v = {lo[0] * il, lo[1] * il, lo[2] * il, lo[3] * il,
                   hi[0] * il, hi[1] * il, hi[2] * il, hi[3] * il};
  *reinterpret_cast<bf16x8*>(a.out + R * DH + grp * 8) = to_bf16x8(v);
}

}  // namespace

hipError_t launch_dense_cache_write(const DenseWriteArgs& a, hipStream_t s) {
  // validated by the caller: d_model % 64 == 0, (2 H d_head) % 128 == 0, d_head even
  const dim3 grid((a.geo.chunk_tokens + kDwTok - 1) / kDwTok, 2 * a.n_heads * a.d_head / kDwOut,
                  a.batch);
  hipLaunchKernelGGL(dense_cache_write_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_dense_q_prep(const AttendArgs& a, hipStream_t s) {
  // validated by the caller: d_v / 2 <= 64 pairs, nq_pad % 4 == 0
  hipLaunchKernelGGL(dense_q_prep_kernel, dim3(a.nq_pad / 4, a.batch), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mat_q_prep(const AttendArgs& a, hipStream_t s) {
  // validated by the caller: dqk_pad = d_nope + d_rope, both even, nq_pad % 4 == 0
  hipLaunchKernelGGL(mat_q_prep_kernel, dim3(a.nq_pad / 4, a.batch), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mat_rope_fill(const AttendArgs& a, uint16_t* kv, hipStream_t s) {
  const int64_t threads = (int64_t)a.batch * a.n_valid * a.n_heads * (a.d_rope / 8);
  hipLaunchKernelGGL(mat_rope_fill_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                     s, a, kv);
  return hipGetLastError();
}

hipError_t launch_dense_merge(const AttendArgs& a, hipStream_t s) {
  const int64_t threads = (int64_t)a.batch * a.geo.q_count * a.n_heads * (a.d_v / 8);
  if (threads >= (int64_t(1) << 32) - 256) return hipErrorInvalidValue;  // 32-bit indices
  hipLaunchKernelGGL(dense_merge_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                     a);
  return hipGetLastError();
}

}  // namespace vmla
