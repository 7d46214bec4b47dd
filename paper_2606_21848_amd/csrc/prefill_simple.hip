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

constexpr int GK = 64;  // k per step: few steps, so few exposed load latencies on small products

// One k-step of the GT x GT output tile: the thread's share of the A tile
// (GT rows x GK columns; consecutive threads take consecutive k) and of the B
// tile (GK rows x GT columns; consecutive threads take consecutive n), zero
// outside the matrices.
template <typename T, int GT>
__device__ __forceinline__ void gemm_load(const GemmParams& p, const T* A, const T* Bm, int m0,
                                          int n0, int k0, size_t acs, size_t bcs,
                                          float (&ra)[GT * GK / 256], float (&rb)[GT * GK / 256]) {
#pragma unroll
  for (int r = 0; r < GT * GK / 256; ++r) {
    const int i = threadIdx.x + 256 * r;
    const int kk = i % GK, mm = i / GK;
    const int gm = m0 + mm, gk = k0 + kk;
    ra[r] = (gm < p.M && gk < p.K) ? ld(A, (size_t)gm * p.lda + gk * acs) : 0.f;
    const int nn = i % GT, kb = i / GT;
    const int gn = n0 + nn, gkb = k0 + kb;
    rb[r] = (gn < p.N && gkb < p.K) ? ld(Bm, (size_t)gkb * p.ldb + gn * bcs) : 0.f;
  }
}

// GT x GT output tile per workgroup of 256 threads (16 x 16 threads, each
// GT / 16 x GT / 16 outputs): 64 for large products, 32 where 64-wide tiles
// would leave most of the chip idle.
template <typename T, int GT>
__global__ __launch_bounds__(256) void gemm_simple_kernel(GemmParams p) {
  constexpr int R = GT / 16, NL = GT * GK / 256;
  const T* A = reinterpret_cast<const T*>(p.A) + (size_t)blockIdx.z * p.strideA;
  const T* Bm = reinterpret_cast<const T*>(p.Bm) + (size_t)blockIdx.z * p.strideB;
  T* C = reinterpret_cast<T*>(p.C) + (size_t)blockIdx.z * p.strideC;
  __shared__ float sA[GK][GT + 1];
  __shared__ float sB[GK][GT + 1];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int m0 = blockIdx.y * GT, n0 = blockIdx.x * GT;
  float c[R][R] = {};
  const size_t acs = p.a_cs ? p.a_cs : 1, bcs = p.b_cs ? p.b_cs : 1;
  // The next k-step's elements are loaded into registers while the current
  // one is multiplied out of LDS.
  float ra[NL], rb[NL];
  gemm_load<T, GT>(p, A, Bm, m0, n0, 0, acs, bcs, ra, rb);
  for (int k0 = 0; k0 < p.K; k0 += GK) {
#pragma unroll
    for (int r = 0; r < NL; ++r) {
      const int i = threadIdx.x + 256 * r;
      sA[i % GK][i / GK] = ra[r];
      sB[i / GT][i % GT] = rb[r];
    }
    __syncthreads();
    if (k0 + GK < p.K) gemm_load<T, GT>(p, A, Bm, m0, n0, k0 + GK, acs, bcs, ra, rb);
#pragma unroll 16
    for (int kk = 0; kk < GK; ++kk) {
      float a[R], bv[R];
#pragma unroll
      for (int i = 0; i < R; ++i) a[i] = sA[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < R; ++j) bv[j] = sB[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < R; ++i)
#pragma unroll
        for (int j = 0; j < R; ++j) c[i][j] = fmaf(a[i], bv[j], c[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int j = 0; j < R; ++j) {
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
    // Four value rows per update: four independent score chains, one rescale.
    // Rows past what this group sees (or past the tile's end) get no weight,
    // and their values are replaced by zeros so that nothing non-finite in them
    // can reach the sum.
    const int jn = min(SV_ROWS, jend - j0);
    for (int jj = 0; jj < jn; jj += 4) {
      f32xE v[4];
      float s[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v[u] = *reinterpret_cast<const f32xE*>(&sV[jj + u][c * E]);
        s[u] = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) s[u] = fmaf(q[e], v[u][e], s[u]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        s[u] = group_sum<16>(s[u]);
        if (j0 + jj + u >= seen || jj + u >= jn) {
          s[u] = -INFINITY;
          v[u] = f32xE{};
        }
      }
      const float mn = fmaxf(fmaxf(m, fmaxf(s[0], s[1])), fmaxf(s[2], s[3]));
      const float ms = mn == -INFINITY ? 0.f : mn;  // nothing seen yet: no shift
      const float alpha = fast_exp2(m - ms);
      float w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) w[u] = fast_exp2(s[u] - ms);
      l = fmaf(l, alpha, (w[0] + w[1]) + (w[2] + w[3]));
#pragma unroll
      for (int e = 0; e < E; ++e)
        acc[e] = fmaf(w[3], v[3][e], fmaf(w[2], v[2][e], fmaf(w[1], v[1][e], fmaf(w[0], v[0][e], acc[e] * alpha))));
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

template <int GT>
hipError_t launch_gemm_gt(const GemmParams& p, hipStream_t st) {
  dim3 grid((p.N + GT - 1) / GT, (p.M + GT - 1) / GT, p.batch);
  if (p.dtype == KL_BF16)
    hipLaunchKernelGGL((gemm_simple_kernel<uint16_t, GT>), grid, dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL((gemm_simple_kernel<float, GT>), grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_gemm_simple(const GemmParams& p, hipStream_t st) {
  if (p.M == 0 || p.N == 0 || p.batch == 0) return hipSuccess;
  const long tiles64 = (long)((p.N + 63) / 64) * ((p.M + 63) / 64) * p.batch;
  return tiles64 < 256 ? launch_gemm_gt<32>(p, st) : launch_gemm_gt<64>(p, st);
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
