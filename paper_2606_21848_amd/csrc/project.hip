// Decode-step projections (Section 3): for the current token of each sequence,
// its routed query q~ = x W~^Q (the query of the decode weights) and its value
// v = x W^V (the row that joins the value-only cache), against the weights
// packed once before inference ([W~^Q | W^V] transposed: row n = output column
// n, d_model contiguous). The value rows are written straight into the cache.
//
// The step is bound by the weight bytes: every packed row is read once per 16
// sequences. A workgroup (16 waves) owns 32 rows; wave w takes the k-steps of
// 32 columns w, w + 16, ... and multiplies them with v_mfma_f32_16x16x32_bf16
// (A = the 16 sequences' x fragments, B = the weight rows, both loaded straight
// into registers, 16 bytes per lane); the waves' partial sums are then added in
// LDS in wave order.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

constexpr int kWaves = 16;
constexpr int kRows = 32;      // packed rows (output columns) per workgroup
constexpr int kMaxK = 16384;   // d_model limit (32-bit offsets, and a bounded loop)

__device__ __forceinline__ uint16_t to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

__global__ __launch_bounds__(kWaves * 64) void project_kernel(ProjectParams p) {
  const int n0 = blockIdx.x * kRows;
  const int b0 = blockIdx.y * 16;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int fr = lane & 15, grp = lane >> 4;
  const int nsteps = p.K / 32;
  const int mine = (nsteps - wave + kWaves - 1) / kWaves;  // k-steps of this wave (uniform)

  // Fragments: x rows b0 + fr (clamped; rows past B are never stored) and
  // weight rows n0 + 16 nb + fr (clamped), columns 32 s + 8 grp .. + 7.
  const uint16_t* xr = p.x + (size_t)min(b0 + fr, p.B - 1) * p.ldx + grp * 8;
  const uint16_t* w0 = p.Wp + (size_t)min(n0 + fr, p.N - 1) * p.K + grp * 8;
  const uint16_t* w1 = p.Wp + (size_t)min(n0 + 16 + fr, p.N - 1) * p.K + grp * 8;
  f32x4_t acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  // Chunks of 8 k-steps: all 24 loads of a chunk are in flight before its MFMAs.
  for (int c = 0; c < mine; c += 8) {  // uniform
    u32x4 xa[8], wa[8], wb[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (c + i < mine) {
        const int k = (wave + (c + i) * kWaves) * 32;
        wa[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(w0 + k));
        wb[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(w1 + k));
        xa[i] = *reinterpret_cast<const u32x4*>(xr + k);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (c + i < mine) {
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, xa[i]);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8_t, wa[i]), acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8_t, wb[i]), acc1, 0, 0, 0);
      }
    }
  }

  // Lane holds C[b0 + 4 grp + r][n0 + 16 nb + fr]; sum the waves in order.
  __shared__ float part[kWaves][16][kRows];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    part[wave][grp * 4 + r][fr] = acc0[r];
    part[wave][grp * 4 + r][16 + fr] = acc1[r];
  }
  __syncthreads();
  if (threadIdx.x >= 16 * kRows) return;
  const int bi = threadIdx.x / kRows, ni = threadIdx.x % kRows;
  const int b = b0 + bi, n = n0 + ni;
  if (b >= p.B || n >= p.N) return;
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) s += part[w][bi][ni];
  const uint16_t val = to_bf16(s);
  if (n < p.NQ) {
    p.q_out[(size_t)b * p.ldq + n] = val;
    return;
  }
  const int j = n - p.NQ;
  if (p.v_out) p.v_out[(size_t)b * p.ldv + j] = val;
  if (!p.cache) return;
  // Append at position lengths_before[b]; positions past the capacity, or in a
  // block outside the cache, are dropped (as value_cache_append does).
  const int g = j / p.D, d = j % p.D;
  const int pos = p.lengths_before[b];
  size_t row;
  if (p.paged) {
    const int cap = p.max_blocks << p.block_shift;
    if (pos < 0 || pos >= cap) return;
    const int blk = p.table[(size_t)b * p.max_blocks + (pos >> p.block_shift)];
    if (blk < 0 || blk >= p.num_blocks) return;
    row = (((size_t)blk * p.G + g) << p.block_shift) + (pos & ((1 << p.block_shift) - 1));
  } else {
    if (pos < 0 || pos >= p.L_max) return;
    row = ((size_t)b * p.G + g) * p.L_max + pos;
  }
  p.cache[row * p.D + d] = val;
}

}  // namespace

bool project_supported(int K) { return K >= 32 && K % 32 == 0 && K <= kMaxK; }

hipError_t launch_project(const ProjectParams& p, hipStream_t st) {
  if (p.B <= 0 || p.N <= 0) return hipSuccess;
  if (!project_supported(p.K)) return hipErrorInvalidValue;
  const dim3 grid((p.N + kRows - 1) / kRows, (p.B + 15) / 16);
  hipLaunchKernelGGL(project_kernel, grid, dim3(kWaves * 64), 0, st, p);
  return hipGetLastError();
}

}  // namespace kl
