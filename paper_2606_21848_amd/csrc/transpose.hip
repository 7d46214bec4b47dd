// bf16 transpose through LDS, for the backward pass through the projections:
// the contractions over tokens (X^T dQ~, X^T dV) run on the MFMA GEMM, which
// wants both operands with the contraction (token) index contiguous.
//
// A workgroup moves a 64 x 64 block: 16-byte loads of source rows into an LDS
// tile padded by one element per row (the column reads then fall in distinct
// banks), and 16-byte stores of destination rows. Destination columns past the
// source's rows, up to rows_pad, are written as zeros, so that a contraction
// over the padded length adds nothing.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

constexpr int TB = 64;  // block edge

__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ src,
                                                             long ld_src, int rows, int cols,
                                                             uint16_t* __restrict__ dst,
                                                             long ld_dst, int rows_pad,
                                                             long s_src, long s_dst) {
  __shared__ uint16_t tile[TB][TB + 2];
  src += (size_t)blockIdx.z * s_src;
  dst += (size_t)blockIdx.z * s_dst;
  const int r0 = blockIdx.x * TB, c0 = blockIdx.y * TB;
  const int t = threadIdx.x;
  const bool vec_src = (ld_src & 7) == 0;
  // Source rows r0 .. r0 + 63, columns c0 .. c0 + 63: 8 chunks of 8 per row.
  for (int i = t; i < TB * 8; i += 256) {
    const int rr = i / 8, cc = (i % 8) * 8;
    const int r = r0 + rr, c = c0 + cc;
    uint16_t v[8];
    if (r < rows && vec_src && c + 8 <= cols) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(src + (size_t)r * ld_src + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] = (uint16_t)(x[e] & 0xFFFFu);
        v[2 * e + 1] = (uint16_t)(x[e] >> 16);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        v[e] = (r < rows && c + e < cols) ? src[(size_t)r * ld_src + c + e] : (uint16_t)0;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) tile[rr][cc + e] = v[e];
  }
  __syncthreads();
  // Destination rows c0 .. c0 + 63 (source columns), columns r0 .. r0 + 63.
  const bool vec_dst = (ld_dst & 7) == 0;
  for (int i = t; i < TB * 8; i += 256) {
    const int cc = i / 8, rr = (i % 8) * 8;
    const int c = c0 + cc, r = r0 + rr;
    if (c >= cols || r >= rows_pad) continue;
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = tile[rr + e][cc];  // rows past `rows` were loaded as zero
    uint16_t* d = dst + (size_t)c * ld_dst + r;
    if (vec_dst && r + 8 <= rows_pad) {
      u32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = (uint32_t)v[2 * e] | ((uint32_t)v[2 * e + 1] << 16);
      *reinterpret_cast<u32x4*>(d) = x;
    } else {
      for (int e = 0; e < 8 && r + e < rows_pad; ++e) d[e] = v[e];
    }
  }
}

}  // namespace

hipError_t launch_transpose_bf16(const void* src, long ld_src, int rows, int cols, void* dst,
                                 long ld_dst, int rows_pad, hipStream_t st, int batch, long s_src,
                                 long s_dst) {
  if (rows < 0 || cols < 0 || rows_pad < rows || batch < 0 || batch > 65535)
    return hipErrorInvalidValue;
  if (rows_pad == 0 || cols == 0 || batch == 0) return hipSuccess;
  const dim3 grid((rows_pad + TB - 1) / TB, (cols + TB - 1) / TB, batch);
  hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(256), 0, st,
                     static_cast<const uint16_t*>(src), ld_src, rows, cols,
                     static_cast<uint16_t*>(dst), ld_dst, rows_pad, s_src, s_dst);
  return hipGetLastError();
}

}  // namespace kl
