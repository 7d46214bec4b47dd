// The two small products around a decode over a latent value-only cache
// (Section 3, Eq. 15), per (sequence b, query head h) with the head's expansion
// matrix W_post_h [r, d_k]:
//   absorb:  q*[b, h] = q~[b, h] W_post_h^T     (d_k -> r, before the decode)
//   expand:  out[b, h] = o*[b, h] W_post_h      (r -> d_k, after the decode)
// Both are y = x M with M = W_post_h^T or W_post_h. A workgroup takes one head
// and up to 32 sequences: it stages M in LDS as fp32 laid out [contraction]
// [output] (row pitch n_out + 1, so the transposing stores of the absorb hit
// distinct banks), stages the 32 input vectors, and each thread accumulates one
// output column for 8 or 16 sequences in fp32. The matrices are read once per
// 32 sequences; both products are tiny next to the cache stream they bracket.

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
  if (p.dtype == KL_BF16)
    return p.absorb ? launch_dims<uint16_t, true>(p, st) : launch_dims<uint16_t, false>(p, st);
  return p.absorb ? launch_dims<float, true>(p, st) : launch_dims<float, false>(p, st);
}

}  // namespace kl
