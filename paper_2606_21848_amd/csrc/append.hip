// Value-cache append (Section 3: the new value joins the cache before the
// decode step that reads it). One thread moves one 16-byte slice of a row.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

template <int SLICES>  // 16-byte slices per row
__global__ __launch_bounds__(256) void append_kernel(AppendParams p) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long row = idx / SLICES;
  const int sl = (int)(idx % SLICES);
  if (row >= (long)p.B * p.T * p.G) return;
  const int g = (int)(row % p.G);
  const int t = (int)((row / p.G) % p.T);
  const int b = (int)(row / ((long)p.G * p.T));
  const int pos = p.lengths_before[b] + t;
  size_t dst_row;
  if (p.paged) {
    const int cap = p.max_blocks << p.block_shift;
    if (pos < 0 || pos >= cap) return;
    const int blk = p.table[(size_t)b * p.max_blocks + (pos >> p.block_shift)];
    if (blk < 0 || blk >= p.num_blocks) return;
    dst_row = (((size_t)blk * p.G + g) << p.block_shift) + (pos & ((1 << p.block_shift) - 1));
  } else {
    if (pos < 0 || pos >= p.L_max) return;
    dst_row = ((size_t)b * p.G + g) * p.L_max + pos;
  }
  const uint4* src = reinterpret_cast<const uint4*>(p.values) + (size_t)row * SLICES + sl;
  uint4* dst = reinterpret_cast<uint4*>(p.data) + dst_row * SLICES + sl;
  *dst = *src;
}

}  // namespace

hipError_t launch_append(const AppendParams& p, hipStream_t st) {
  const int row_bytes = p.D * (p.dtype == KL_BF16 ? 2 : 4);
  const int slices = row_bytes / 16;
  const long threads = (long)p.B * p.T * p.G * slices;
  if (threads == 0) return hipSuccess;
  const dim3 grid((unsigned)((threads + 255) / 256));
  switch (slices) {
    case 8: hipLaunchKernelGGL(append_kernel<8>, grid, dim3(256), 0, st, p); break;
    case 16: hipLaunchKernelGGL(append_kernel<16>, grid, dim3(256), 0, st, p); break;
    case 32: hipLaunchKernelGGL(append_kernel<32>, grid, dim3(256), 0, st, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kl
