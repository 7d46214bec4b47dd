// Two measuring kernels that set the practical ceilings the roofline fractions
// are read against on this chip (they are not part of the method): a plain
// streaming read of a buffer, and a loop of independent matrix-core products
// on constant operands.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

constexpr int kProbeThreads = 256;

// Every 16-byte chunk of src once, with non-temporal loads: workgroup w streams
// its own contiguous share of the buffer, 32 KiB per step (eight 16-byte loads
// in flight per lane, each load instruction of a wave covering 1 KiB of
// consecutive addresses). Each lane folds what it read into one word; the word
// is stored only if it equals a constant no input is expected to give, so the
// loads cannot be dropped and nothing else is written.
__global__ __launch_bounds__(kProbeThreads) void probe_read_kernel(const u32x4* __restrict__ src,
                                                                  size_t n, unsigned* sink) {
  const size_t per = (n + gridDim.x - 1) / gridDim.x;  // chunks per workgroup
  const size_t begin = (size_t)blockIdx.x * per;
  const size_t end = begin + per < n ? begin + per : n;
  size_t i = begin + threadIdx.x;
  unsigned a = 0;
  for (; i + 7 * kProbeThreads < end; i += 8 * kProbeThreads) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(src + i + u * kProbeThreads);
#pragma unroll
    for (int u = 0; u < 8; ++u) a ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < end; i += kProbeThreads) {
    const u32x4 v = __builtin_nontemporal_load(src + i);
    a ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (a == 0x9E3779B9u) *sink = a;
}

// Per wave, iters rounds of 16 independent v_mfma_f32_16x16x32_bf16 on constant
// operands; 16 x 16 x 32 x 2 FLOP each. One round is a single asm block with
// each accumulator tied to its own registers, so the loop carries them in place
// (compiled from plain intrinsics, the loop-carried accumulators were moved
// between registers every round). Each accumulator is read again 15 products
// after it was written, past every dependency wait of the matrix pipe.
__global__ __launch_bounds__(kProbeThreads) void probe_mfma_kernel(int iters, float* sink) {
  const bf16x8_t a = {(__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f,
                      (__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f};
  const bf16x8_t b = {(__bf16)0.5f, (__bf16)0.5f, (__bf16)0.5f, (__bf16)0.5f,
                      (__bf16)0.5f, (__bf16)0.5f, (__bf16)0.5f, (__bf16)0.5f};
  f32x4_t c[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) c[j] = f32x4_t{(float)j, 0.f, 0.f, (float)threadIdx.x};
#define KL_PROBE_MFMA(k) "v_mfma_f32_16x16x32_bf16 %" #k ", %16, %17, %" #k "\n\t"
  for (int it = 0; it < iters; ++it) {
    asm volatile(KL_PROBE_MFMA(0) KL_PROBE_MFMA(1) KL_PROBE_MFMA(2) KL_PROBE_MFMA(3)
                 KL_PROBE_MFMA(4) KL_PROBE_MFMA(5) KL_PROBE_MFMA(6) KL_PROBE_MFMA(7)
                 KL_PROBE_MFMA(8) KL_PROBE_MFMA(9) KL_PROBE_MFMA(10) KL_PROBE_MFMA(11)
                 KL_PROBE_MFMA(12) KL_PROBE_MFMA(13) KL_PROBE_MFMA(14) KL_PROBE_MFMA(15)
                 : "+a"(c[0]), "+a"(c[1]), "+a"(c[2]), "+a"(c[3]), "+a"(c[4]), "+a"(c[5]),
                   "+a"(c[6]), "+a"(c[7]), "+a"(c[8]), "+a"(c[9]), "+a"(c[10]), "+a"(c[11]),
                   "+a"(c[12]), "+a"(c[13]), "+a"(c[14]), "+a"(c[15])
                 : "v"(a), "v"(b));
  }
#undef KL_PROBE_MFMA
  // The results are read long after the last product (the pipe drains first).
  __builtin_amdgcn_s_sleep(2);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) s += c[j][0] + c[j][1] + c[j][2] + c[j][3];
  if (s == -1.f) *sink = s;
}

}  // namespace

hipError_t launch_probe_read(const void* src, size_t bytes, unsigned* sink, int workgroups,
                             hipStream_t st) {
  hipLaunchKernelGGL(probe_read_kernel, dim3(workgroups), dim3(kProbeThreads), 0, st,
                     static_cast<const u32x4*>(src), bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_probe_mfma(float* sink, int iters, int workgroups, hipStream_t st) {
  hipLaunchKernelGGL(probe_mfma_kernel, dim3(workgroups), dim3(kProbeThreads), 0, st, iters, sink);
  return hipGetLastError();
}

}  // namespace kl
