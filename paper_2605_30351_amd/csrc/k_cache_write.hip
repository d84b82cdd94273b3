// Fused cache write: compress (Eq. 1), optional RMSNorm of the latent, decoupled RoPE key
// (Eq. 5) rotated at the token's absolute (f, y, x) (kept unrotated when the cache has an
// attention sink, Sec. "Decoupled 3D-RoPE"), and FIFO placement into the ring.
//
// One workgroup takes 32 chunk tokens of one batch element and all d_c + d_rope outputs:
// out^T[o][token] = W[o][:] . x[token][:] with MFMA 32x32x16 (A = rows of [W_DKV; W_KR],
// B = x rows). The contraction over d_model streams through a ring of kStages LDS stages of
// kKC columns each, filled by direct global-to-LDS loads (no registers, several chunks in
// flight) in an XOR-swizzled layout that makes the MFMA operand reads conflict-free. The four
// waves share every staged chunk and split the 32-row output blocks between them. The epilogue
// combines the RMSNorm sum of squares across waves in LDS, normalizes, rotates the RoPE block,
// rounds to bf16 and stores each token's values to its ring slot.
#include "vmla_device.h"

namespace vmla {
namespace {

constexpr int kTok = 32;     // tokens per workgroup
constexpr int kWaves = 4;
constexpr int kKC = 64;      // contraction columns per stage: 8 chunks of 16 B per row

// Position (16 B units) of chunk c of staged row r: row-major with 8 chunks per row, the chunk
// index XOR-ed with (r / 2) mod 8, so 16 consecutive rows read at one chunk hit distinct banks.
__device__ __forceinline__ int swz(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

template <int NB>  // 32-wide output blocks covering d_c + d_rope
__global__ __launch_bounds__(kWaves * 64) void cache_write_kernel(const WriteArgs a) {
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
          rope_rotate(a.rope, ch / 2, pos, v[0], v[1]);
          rope_rotate(a.rope, ch / 2 + 1, pos, v[2], v[3]);
        }
        const f32x4 fv = {v[0], v[1], v[2], v[3]};
        *reinterpret_cast<bf16x4*>(kdst + ch) = to_bf16x4(fv);
      }
    }
  }
  if (a.slots && b == 0 && wave == 0 && g == 0) a.slots[n] = (int32_t)slot;
}

}  // namespace

hipError_t launch_cache_write(const WriteArgs& a, hipStream_t s) {
  // validated by the caller: d_model % 64 == 0, d_c % 16 == 0, d_rope % 8 == 0,
  // d_c + d_rope <= 288
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
