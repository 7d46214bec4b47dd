// The two small products around a decode over a latent value-only cache
// (Section 3, Eq. 15), per (sequence b, query head h) with the head's expansion
// matrix W_post_h [r, d_k]:
//   absorb:  q*[b, h] = q~[b, h] W_post_h^T     (d_k -> r, before the decode)
//   expand:  out[b, h] = o*[b, h] W_post_h      (r -> d_k, after the decode)
// Both are y = x M with M = W_post_h^T or W_post_h, tiny next to the cache
// stream they bracket, so they are built for latency: bf16 runs one wave per
// (head, 16 sequences, 64 output columns) on v_mfma_f32_16x16x32_bf16 with
// both operands loaded straight into registers (the absorb's weight fragments
// are 16-byte row pieces of W_post_h; the expand's are 8 column elements,
// loaded 2 bytes at a time, 16 lanes covering 32 contiguous bytes). fp32 runs
// a VALU kernel: a workgroup takes one head and up to 32 sequences, stages M
// in LDS as [contraction][output] (row pitch n_out + 1, so the transposing
// stores of the absorb hit distinct banks) and each thread accumulates one
// output column for 8 or 16 sequences.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

constexpr int kSeq = 32;       // sequences per workgroup
constexpr int kThreads = 256;

template <typename T>
__device__ __forceinline__ float ldf(const T* p, size_t i) {
  if constexpr (sizeof(T) == 2) return __uint_as_float((uint32_t)p[i] << 16);
  else return p[i];
}

template <typename T>
__device__ __forceinline__ void stf(T* p, size_t i, float v) {
  if constexpr (sizeof(T) == 2) p[i] = __builtin_bit_cast(uint16_t, (__bf16)v);
  else p[i] = v;
}

// NIN: contraction length, NOUT: output length (64 or 128 each).
template <typename T, int NIN, int NOUT, bool ABSORB>
__global__ __launch_bounds__(kThreads) void latent_product_kernel(LatentParams p) {
  constexpr int PITCH = NOUT + 1;
  constexpr int NSUB = kThreads / NOUT;   // sequence subsets
  constexpr int PER = kSeq / NSUB;        // sequences per thread
  __shared__ float sM[NIN * PITCH];
  __shared__ float sX[kSeq][NIN];
  const int h = blockIdx.x;
  const int b0 = blockIdx.y * kSeq;
  const int t = threadIdx.x;
  const T* W = reinterpret_cast<const T*>(p.W) + (size_t)h * p.r * p.dk;
  // W_post_h is [r][d_k] row-major. Absorb contracts over d_k: sM[c][j] = W[j][c].
  // Expand contracts over r: sM[j][c] = W[j][c].
  for (int i = t; i < NIN * NOUT; i += kThreads) {
    const int row = i / p.dk, col = i % p.dk;  // element W[row][col], read in order
    const float w = ldf(W, i);
    if constexpr (ABSORB) sM[col * PITCH + row] = w;
    else sM[row * PITCH + col] = w;
  }
  const T* X = reinterpret_cast<const T*>(p.x);
  for (int i = t; i < kSeq * NIN; i += kThreads) {
    const int bi = i / NIN, k = i % NIN;
    const int b = b0 + bi;
    sX[bi][k] = b < p.B ? ldf(X, ((size_t)b * p.H + h) * NIN + k) : 0.f;
  }
  __syncthreads();
  const int n = t % NOUT, sub = t / NOUT;
  float acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) acc[i] = 0.f;
#pragma unroll 4
  for (int k = 0; k < NIN; ++k) {
    const float m = sM[k * PITCH + n];
#pragma unroll
    for (int i = 0; i < PER; ++i) acc[i] = fmaf(sX[sub + i * NSUB][k], m, acc[i]);
  }
  T* Y = reinterpret_cast<T*>(p.y);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int b = b0 + sub + i * NSUB;
    if (b < p.B) stf(Y, ((size_t)b * p.H + h) * NOUT + n, acc[i]);
  }
}

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// bf16: y[b, h, n] for b in [16 by, +16), n in [64 bz, +64); NIN, NOUT in {64, 128}.
template <int NIN, int NOUT, bool ABSORB>
__global__ __launch_bounds__(64) void latent_mfma_kernel(LatentParams p) {
  const int h = blockIdx.x, b0 = blockIdx.y * 16, n0 = blockIdx.z * 64;
  const int lane = threadIdx.x, fr = lane & 15, grp = lane >> 4;
  const uint16_t* __restrict__ X = reinterpret_cast<const uint16_t*>(p.x);
  const uint16_t* __restrict__ W = reinterpret_cast<const uint16_t*>(p.W) + (size_t)h * p.r * p.dk;
  // A operand: x row b0 + fr (clamped; rows past B are never stored), k = 32 ks + 8 grp .. + 7.
  const uint16_t* xrow = X + ((size_t)min(b0 + fr, p.B - 1) * p.H + h) * NIN + 8 * grp;
  f32x4_t acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < NIN / 32; ++ks) {
    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(xrow + 32 * ks));
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int n = n0 + 16 * nb + fr;  // output column of this lane
      const int k0 = 32 * ks + 8 * grp;
      u32x4 w;
      if constexpr (ABSORB) {
        // M[k][n] = W_post_h[n][k]: eight consecutive k of row n.
        w = *reinterpret_cast<const u32x4*>(W + (size_t)n * NIN + k0);
      } else {
        // M[k][n] = W_post_h[k][n]: column n, rows k0 .. k0 + 7.
#pragma unroll
        for (int i = 0; i < 4; ++i)
          w[i] = (uint32_t)W[(size_t)(k0 + 2 * i) * NOUT + n] |
                 ((uint32_t)W[(size_t)(k0 + 2 * i + 1) * NOUT + n] << 16);
      }
      acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8_t, w),
                                                        acc[nb], 0, 0, 0);
    }
  }
  // Lane holds y[b0 + 4 grp + i][n0 + 16 nb + fr].
  uint16_t* __restrict__ Y = reinterpret_cast<uint16_t*>(p.y);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int b = b0 + 4 * grp + i;
    if (b >= p.B) continue;
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      Y[((size_t)b * p.H + h) * NOUT + n0 + 16 * nb + fr] =
          __builtin_bit_cast(uint16_t, (__bf16)acc[nb][i]);
  }
}

template <bool ABSORB>
hipError_t launch_mfma(const LatentParams& p, hipStream_t st) {
  const int nin = ABSORB ? p.dk : p.r, nout = ABSORB ? p.r : p.dk;
  const dim3 grid(p.H, (p.B + 15) / 16, nout / 64);
  if (nin == 128 && nout == 128)
    hipLaunchKernelGGL((latent_mfma_kernel<128, 128, ABSORB>), grid, dim3(64), 0, st, p);
  else if (nin == 128 && nout == 64)
    hipLaunchKernelGGL((latent_mfma_kernel<128, 64, ABSORB>), grid, dim3(64), 0, st, p);
  else if (nin == 64 && nout == 128)
    hipLaunchKernelGGL((latent_mfma_kernel<64, 128, ABSORB>), grid, dim3(64), 0, st, p);
  else
    hipLaunchKernelGGL((latent_mfma_kernel<64, 64, ABSORB>), grid, dim3(64), 0, st, p);
  return hipGetLastError();
}

template <typename T, bool ABSORB>
hipError_t launch_dims(const LatentParams& p, hipStream_t st) {
  const dim3 grid(p.H, (p.B + kSeq - 1) / kSeq);
  const int nin = ABSORB ? p.dk : p.r, nout = ABSORB ? p.r : p.dk;
  if (nin == 128 && nout == 128)
    hipLaunchKernelGGL((latent_product_kernel<T, 128, 128, ABSORB>), grid, dim3(kThreads), 0, st, p);
  else if (nin == 128 && nout == 64)
    hipLaunchKernelGGL((latent_product_kernel<T, 128, 64, ABSORB>), grid, dim3(kThreads), 0, st, p);
  else if (nin == 64 && nout == 128)
    hipLaunchKernelGGL((latent_product_kernel<T, 64, 128, ABSORB>), grid, dim3(kThreads), 0, st, p);
  else if (nin == 64 && nout == 64)
    hipLaunchKernelGGL((latent_product_kernel<T, 64, 64, ABSORB>), grid, dim3(kThreads), 0, st, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_latent_product(const LatentParams& p, hipStream_t st) {
  if (p.B <= 0 || p.H <= 0) return hipSuccess;
  if ((p.r != 64 && p.r != 128) || (p.dk != 64 && p.dk != 128)) return hipErrorInvalidValue;
  if (p.dtype == KL_BF16) return p.absorb ? launch_mfma<true>(p, st) : launch_mfma<false>(p, st);
  return p.absorb ? launch_dims<float, true>(p, st) : launch_dims<float, false>(p, st);
}

}  // namespace kl
