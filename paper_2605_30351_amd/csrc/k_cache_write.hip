// Fused cache write: compress (Eq. 1), optional RMSNorm of the latent, decoupled RoPE key
// (Eq. 5) rotated at the token's absolute (f, y, x), and FIFO placement into the ring.
//
// One workgroup takes 32 chunk tokens of one batch element and all d_c + d_rope outputs. The
// contraction over d_model is split four ways across the waves, so x is read once per
// workgroup and the weight panel once per workgroup. Each wave computes
// out^T[o][token] = W[o][:] . x[token][:] with MFMA 32x32x16 (A = weight rows, B = x rows), the
// four partial products are summed in LDS, and the epilogue normalizes, rotates, rounds to bf16
// and scatters each token's row to its ring slot with 16-byte stores.
#include "vmla_device.h"

namespace vmla {
namespace {

constexpr int kTok = 32;      // tokens per workgroup
constexpr int kWaves = 4;     // waves per workgroup (split of the d_model contraction)

template <int NB>  // 32-wide output blocks covering d_c + d_rope
__global__ __launch_bounds__(kWaves * 64) void cache_write_kernel(const WriteArgs a) {
  constexpr int OUT_STRIDE = NB * 32 + 4;
  __shared__ __attribute__((aligned(16))) float red[kTok][OUT_STRIDE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int b = blockIdx.y;
  const int n0 = blockIdx.x * kTok;
  const int dm = a.d_model, DC = a.d_c, DR = a.d_rope;
  const int n_tok = a.geo.chunk_tokens;

  // A operand rows: output o = ob*32 + l32 reads row o of [W_DKV; W_KR] (zero past the end).
  const uint16_t* wrow[NB];
#pragma unroll
  for (int ob = 0; ob < NB; ++ob) {
    const int o = ob * 32 + l32;
    wrow[ob] = o < DC ? a.w_dkv + (size_t)o * dm
                      : (o < DC + DR ? a.w_kr + (size_t)(o - DC) * dm : nullptr);
  }
  const int n_mine = n0 + l32;
  const bool tok_ok = n_mine < n_tok;
  const uint16_t* xrow = a.x + ((size_t)b * n_tok + (tok_ok ? n_mine : 0)) * dm;

  f32x16 acc[NB];
#pragma unroll
  for (int ob = 0; ob < NB; ++ob) acc[ob] = f32x16{};

  const int kq = dm / kWaves;
  const int kb = wave * kq;
  const u32x4 zero = {0, 0, 0, 0};
#pragma unroll 2
  for (int k = kb; k < kb + kq; k += 16) {
    const bf16x8 bx = as_bf16x8(tok_ok ? ldg16(xrow + k + g * 8) : zero);
#pragma unroll
    for (int ob = 0; ob < NB; ++ob) {
      const bf16x8 aw = as_bf16x8(wrow[ob] ? ldg16(wrow[ob] + k + g * 8) : zero);
      acc[ob] = mfma32(aw, bx, acc[ob]);
    }
  }

  // Sum the four partial products in LDS, one wave at a time.
#pragma unroll 1
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int ob = 0; ob < NB; ++ob) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f32x4* dst = reinterpret_cast<f32x4*>(&red[l32][ob * 32 + 8 * i + 4 * g]);
          const f32x4 v = {acc[ob][4 * i], acc[ob][4 * i + 1], acc[ob][4 * i + 2], acc[ob][4 * i + 3]};
          *dst = w == 0 ? v : *dst + v;
        }
      }
    }
    __syncthreads();
  }

  // Epilogue: 8 threads per token.
  const int tok = tid >> 3, sub = tid & 7;
  const int n = n0 + tok;
  const int oct_c = DC / 8;
  float ss = 0.f;
  for (int ch = sub; ch < oct_c; ch += 8) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float v = red[tok][ch * 8 + e];
      ss += v * v;
    }
  }
  ss += __shfl_xor(ss, 1, 8);
  ss += __shfl_xor(ss, 2, 8);
  ss += __shfl_xor(ss, 4, 8);
  const float rstd = a.gamma ? rsqrtf(ss / (float)DC + a.eps) : 1.f;
  if (n >= n_tok) return;

  const TokenPos pos = token_pos(a.geo, n);
  const int64_t slot = ring_slot(a.geo, pos);
  uint16_t* cdst = a.c_kv + ((size_t)b * a.geo.ring_tokens + slot) * DC;
  for (int ch = sub; ch < oct_c; ch += 8) {
    f32x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float c = red[tok][ch * 8 + e] * rstd;
      if (a.gamma) c *= bf16_bits_to_f32(a.gamma[ch * 8 + e]);
      v[e] = c;
    }
    stg16(cdst + ch * 8, as_u32x4(to_bf16x8(v)));
  }
  uint16_t* kdst = a.k_r + ((size_t)b * a.geo.ring_tokens + slot) * DR;
  for (int p = sub; p < DR / 2; p += 8) {
    float u = red[tok][DC + 2 * p], v = red[tok][DC + 2 * p + 1];
    rope_rotate(a.rope, p, pos, u, v);
    const uint32_t packed = (uint32_t)to_bf16_bits(u) | ((uint32_t)to_bf16_bits(v) << 16);
    *reinterpret_cast<uint32_t*>(kdst + 2 * p) = packed;
  }
  if (a.slots && b == 0 && sub == 0) a.slots[n] = (int32_t)slot;
}

}  // namespace

hipError_t launch_cache_write(const WriteArgs& a, hipStream_t s) {
  const int nb = (a.d_c + a.d_rope + 31) / 32;
  const dim3 grid((a.geo.chunk_tokens + kTok - 1) / kTok, a.batch);
  const dim3 block(kWaves * 64);
  switch (nb) {
    case 1: hipLaunchKernelGGL(cache_write_kernel<1>, grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL(cache_write_kernel<2>, grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL(cache_write_kernel<3>, grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL(cache_write_kernel<4>, grid, block, 0, s, a); break;
    case 5: hipLaunchKernelGGL(cache_write_kernel<5>, grid, block, 0, s, a); break;
    case 6: hipLaunchKernelGGL(cache_write_kernel<6>, grid, block, 0, s, a); break;
    case 7: hipLaunchKernelGGL(cache_write_kernel<7>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(cache_write_kernel<8>, grid, block, 0, s, a); break;
    case 9: hipLaunchKernelGGL(cache_write_kernel<9>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace vmla
