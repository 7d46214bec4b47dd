// Generic (VALU, fp32 arithmetic) kernels for the small products and the fp32
// prefill: a tiled GEMM used for the routing fold W~^Q_h = W^Q_h W^R_h, the fp32
// projections and the weight gradients, and a flash-style keyless attention
// where one LDS tile of values serves both the scores (Eq. 4) and the weighted
// sum. Both are shaped for latency on small problems (the fp32 layer of a few
// hundred tokens): 64-wide k-steps with the next step's loads in flight, and
// 16 lanes per query row.

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

constexpr int GT = 64;  // output tile (64 x 64, 4 x 4 per thread)
constexpr int GK = 64;  // k per step: few steps, so few exposed load latencies on small products

// The 16 A and 16 B elements one thread stages per k-step: A is GT rows x GK
// columns (consecutive threads take consecutive k), B is GK rows x GT columns
// (consecutive threads take consecutive n), zero outside the matrices.
template <typename T>
__device__ __forceinline__ void gemm_load(const GemmParams& p, const T* A, const T* Bm, int m0,
                                          int n0, int k0, size_t acs, size_t bcs, float (&ra)[16],
                                          float (&rb)[16]) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = threadIdx.x + 256 * r;
    const int kk = i % GK, mm = i / GK;
    const int gm = m0 + mm, gk = k0 + kk;
    ra[r] = (gm < p.M && gk < p.K) ? ld(A, (size_t)gm * p.lda + gk * acs) : 0.f;
    const int nn = i % GT, kb = i / GT;
    const int gn = n0 + nn, gkb = k0 + kb;
    rb[r] = (gn < p.N && gkb < p.K) ? ld(Bm, (size_t)gkb * p.ldb + gn * bcs) : 0.f;
  }
}

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
  // The next k-step's elements are loaded into registers while the current
  // one is multiplied out of LDS.
  float ra[16], rb[16];
  gemm_load<T>(p, A, Bm, m0, n0, 0, acs, bcs, ra, rb);
  for (int k0 = 0; k0 < p.K; k0 += GK) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = threadIdx.x + 256 * r;
      sA[i % GK][i / GK] = ra[r];
      sB[i / GT][i % GT] = rb[r];
    }
    __syncthreads();
    if (k0 + GK < p.K) gemm_load<T>(p, A, Bm, m0, n0, k0 + GK, acs, bcs, ra, rb);
#pragma unroll 16
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

// Vector-ALU attention (fp32, and bf16 where the matrix-core kernel does not
// apply). A workgroup of 4 waves owns 16 query rows of one head; each query row
// has 16 lanes, lane c holding columns c E .. c E + E - 1 (E = D / 16) of the
// routed query and of the running output. Value tiles of 64 rows are staged in
// LDS once and serve both the scores (Eq. 4) and the weighted sum; a score is
// the lanes' partial dot products summed over the 16 lanes, and the online
// softmax (m, l, acc) is updated once per value row.
constexpr int SQ_ROWS = 16;  // query rows per workgroup
constexpr int SV_ROWS = 64;  // value rows per staged tile

template <typename T, int D>
__global__ __launch_bounds__(256) void attn_simple_kernel(AttnParams p) {
  constexpr int E = D / 16;
  typedef float f32xE __attribute__((ext_vector_type(E)));
  const int i0 = blockIdx.x * SQ_ROWS;
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (p.H / p.G);
  const int t = threadIdx.x, c = t & 15;
  const int i = i0 + (t >> 4);  // this lane group's query row
  const T* Q = reinterpret_cast<const T*>(p.q);
  const T* V = reinterpret_cast<const T*>(p.v);
  __shared__ __attribute__((aligned(16))) float sV[SV_ROWS][D];
  const bool live = i < p.N;
  f32xE q, acc;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    q[e] = live ? ld(Q, ((size_t)b * p.N + i) * p.q_stride + (size_t)h * D + c * E + e) * p.scale_log2
                : 0.f;
    acc[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  // Rows this lane group sees, and the rows any group of the workgroup sees.
  const int seen = live ? (p.causal ? min(i + 1, p.Nk) : p.Nk) : 0;
  const int jend = p.causal ? min(p.Nk, min(p.N, i0 + SQ_ROWS)) : p.Nk;
  for (int j0 = 0; j0 < jend; j0 += SV_ROWS) {
    __syncthreads();
    for (int e = t; e < SV_ROWS * D; e += 256) {
      const int jj = e / D, cc = e % D;
      const int j = j0 + jj;
      sV[jj][cc] = (j < p.Nk) ? ld(V, ((size_t)b * p.Nk + j) * p.v_stride + (size_t)g * D + cc) : 0.f;
    }
    __syncthreads();
    const int jn = min(SV_ROWS, jend - j0);
    for (int jj = 0; jj < jn; ++jj) {
      const f32xE v = *reinterpret_cast<const f32xE*>(&sV[jj][c * E]);
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) s = fmaf(q[e], v[e], s);
      s = group_sum<16>(s);
      if (j0 + jj >= seen) s = -INFINITY;
      const float mn = fmaxf(m, s);
      const float ms = mn == -INFINITY ? 0.f : mn;  // nothing seen yet: no shift
      const float alpha = fast_exp2(m - ms), w = fast_exp2(s - ms);
      l = fmaf(l, alpha, w);
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(w, v[e], acc[e] * alpha);
      m = mn;
    }
  }
  if (live) {
    T* O = reinterpret_cast<T*>(p.out);
    const float inv = l > 0.f ? 1.f / l : 0.f;  // no value rows: a zero row
    if (p.lse && c == 0)  // m and the scores are in log2 units
      p.lse[((size_t)b * p.H + h) * p.N + i] =
          l > 0.f ? (m + __log2f(l)) * 0.69314718055994531f : -INFINITY;
#pragma unroll
    for (int e = 0; e < E; ++e)
      st(O, ((size_t)b * p.N + i) * p.o_stride + (size_t)h * D + c * E + e, acc[e] * inv);
    if (p.out_f32) {
#pragma unroll
      for (int e = 0; e < E; ++e)
        p.out_f32[(((size_t)b * p.N + i) * p.H + h) * D + c * E + e] = acc[e] * inv;
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
  dim3 grid((p.N + SQ_ROWS - 1) / SQ_ROWS, p.H, p.B);
  if (p.dtype == KL_BF16) {
    if (p.D == 64) hipLaunchKernelGGL((attn_simple_kernel<uint16_t, 64>), grid, dim3(256), 0, st, p);
    else if (p.D == 128) hipLaunchKernelGGL((attn_simple_kernel<uint16_t, 128>), grid, dim3(256), 0, st, p);
    else return hipErrorInvalidValue;
  } else {
    if (p.D == 64) hipLaunchKernelGGL((attn_simple_kernel<float, 64>), grid, dim3(256), 0, st, p);
    else if (p.D == 128) hipLaunchKernelGGL((attn_simple_kernel<float, 128>), grid, dim3(256), 0, st, p);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kl
