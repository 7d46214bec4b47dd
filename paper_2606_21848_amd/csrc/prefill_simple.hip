// Generic (VALU, fp32 arithmetic) kernels for the small products and the fp32
// prefill: a tiled GEMM used for the routing fold W~^Q_h = W^Q_h W^R_h and for
// the fp32 projections, and a flash-style causal keyless attention where one
// LDS tile of values serves both the scores (Eq. 4) and the weighted sum.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

template <typename T>
__device__ __forceinline__ float ld(const T* p, size_t i);
template <>
__device__ __forceinline__ float ld<float>(const float* p, size_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ld<uint16_t>(const uint16_t* p, size_t i) {
  return __uint_as_float((uint32_t)p[i] << 16);
}
template <typename T>
__device__ __forceinline__ void st(T* p, size_t i, float v);
template <>
__device__ __forceinline__ void st<float>(float* p, size_t i, float v) { p[i] = v; }
template <>
__device__ __forceinline__ void st<uint16_t>(uint16_t* p, size_t i, float v) {
  p[i] = (uint16_t)f32_to_bf16(v);
}

constexpr int GT = 64;  // output tile
constexpr int GK = 16;  // k step

template <typename T>
__global__ __launch_bounds__(256) void gemm_simple_kernel(GemmParams p) {
  const T* A = reinterpret_cast<const T*>(p.A) + (size_t)blockIdx.z * p.strideA;
  const T* Bm = reinterpret_cast<const T*>(p.Bm) + (size_t)blockIdx.z * p.strideB;
  T* C = reinterpret_cast<T*>(p.C) + (size_t)blockIdx.z * p.strideC;
  __shared__ float sA[GK][GT + 1];
  __shared__ float sB[GK][GT + 1];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int m0 = blockIdx.y * GT, n0 = blockIdx.x * GT;
  float c[4][4] = {};
  const size_t acs = p.a_cs ? p.a_cs : 1, bcs = p.b_cs ? p.b_cs : 1;
  for (int k0 = 0; k0 < p.K; k0 += GK) {
    for (int i = threadIdx.x; i < GK * GT; i += 256) {
      const int kk = i % GK, mm = i / GK;  // A tile: GT rows x GK cols
      const int gm = m0 + mm, gk = k0 + kk;
      sA[kk][mm] = (gm < p.M && gk < p.K) ? ld(A, (size_t)gm * p.lda + gk * acs) : 0.f;
      const int nn = i % GT, kb = i / GT;  // B tile: GK rows x GT cols
      const int gn = n0 + nn, gkb = k0 + kb;
      sB[kb][nn] = (gn < p.N && gkb < p.K) ? ld(Bm, (size_t)gkb * p.ldb + gn * bcs) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GK; ++kk) {
      float a[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = sB[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) c[i][j] = fmaf(a[i], bv[j], c[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int gm = m0 + ty + 16 * i, gn = n0 + tx + 16 * j;
      if (gm < p.M && gn < p.N) {
        const size_t at = (size_t)gm * p.ldc + gn;
        st(C, at, p.accumulate ? ld(reinterpret_cast<const T*>(C), at) + c[i][j] : c[i][j]);
      }
    }
}

// One thread per query row; 64 query rows per workgroup. Value tiles of 64 rows
// are staged in LDS once and read by every thread for both uses.
template <typename T, int D>
__global__ __launch_bounds__(64) void attn_simple_kernel(AttnParams p) {
  const int i0 = blockIdx.x * 64;
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (p.H / p.G);
  const int i = i0 + threadIdx.x;
  const T* Q = reinterpret_cast<const T*>(p.q);
  const T* V = reinterpret_cast<const T*>(p.v);
  __shared__ float sV[64][D];
  float q[D], acc[D];
  const bool live = i < p.N;
#pragma unroll
  for (int c = 0; c < D; ++c) {
    q[c] = live ? ld(Q, ((size_t)b * p.N + i) * p.q_stride + (size_t)h * D + c) * p.scale_log2 : 0.f;
    acc[c] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int jend = p.causal ? min(p.Nk, i0 + 64) : p.Nk;
  for (int j0 = 0; j0 < jend; j0 += 64) {
    __syncthreads();
    for (int e = threadIdx.x; e < 64 * D; e += 64) {
      const int jj = e / D, c = e % D;
      const int j = j0 + jj;
      sV[jj][c] = (j < p.Nk) ? ld(V, ((size_t)b * p.Nk + j) * p.v_stride + (size_t)g * D + c) : 0.f;
    }
    __syncthreads();
    const int jmax = min(64, (p.causal ? min(i + 1, p.Nk) : p.Nk) - j0);
    for (int jj = 0; jj < jmax; ++jj) {
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) s = fmaf(q[c], sV[jj][c], s);
      const float mn = fmaxf(m, s);
      const float alpha = fast_exp2(m - mn);
      const float w = fast_exp2(s - mn);
      l = l * alpha + w;
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = fmaf(w, sV[jj][c], acc[c] * alpha);
      m = mn;
    }
  }
  if (live) {
    T* O = reinterpret_cast<T*>(p.out);
    const float inv = l > 0.f ? 1.f / l : 0.f;  // no value rows: a zero row
    if (p.lse)  // m and the scores are in log2 units
      p.lse[((size_t)b * p.H + h) * p.N + i] =
          l > 0.f ? (m + __log2f(l)) * 0.69314718055994531f : -INFINITY;
#pragma unroll
    for (int c = 0; c < D; ++c) st(O, ((size_t)b * p.N + i) * p.o_stride + (size_t)h * D + c, acc[c] * inv);
    if (p.out_f32) {
#pragma unroll
      for (int c = 0; c < D; ++c) p.out_f32[(((size_t)b * p.N + i) * p.H + h) * D + c] = acc[c] * inv;
    }
  }
}

}  // namespace

hipError_t launch_gemm_simple(const GemmParams& p, hipStream_t st) {
  if (p.M == 0 || p.N == 0 || p.batch == 0) return hipSuccess;
  dim3 grid((p.N + GT - 1) / GT, (p.M + GT - 1) / GT, p.batch);
  if (p.dtype == KL_BF16)
    hipLaunchKernelGGL(gemm_simple_kernel<uint16_t>, grid, dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(gemm_simple_kernel<float>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_prefill_attention_simple(const AttnParams& p, hipStream_t st) {
  if (p.N == 0 || p.B == 0) return hipSuccess;
  if (p.Nk < 0 || (p.causal && p.Nk != p.N)) return hipErrorInvalidValue;
  dim3 grid((p.N + 63) / 64, p.H, p.B);
  if (p.dtype == KL_BF16) {
    if (p.D == 64) hipLaunchKernelGGL((attn_simple_kernel<uint16_t, 64>), grid, dim3(64), 0, st, p);
    else if (p.D == 128) hipLaunchKernelGGL((attn_simple_kernel<uint16_t, 128>), grid, dim3(64), 0, st, p);
    else return hipErrorInvalidValue;
  } else {
    if (p.D == 64) hipLaunchKernelGGL((attn_simple_kernel<float, 64>), grid, dim3(64), 0, st, p);
    else if (p.D == 128) hipLaunchKernelGGL((attn_simple_kernel<float, 128>), grid, dim3(64), 0, st, p);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kl
