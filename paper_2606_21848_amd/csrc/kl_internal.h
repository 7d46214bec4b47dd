// Internal launch interface between the C-ABI host code and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "keyless.h"

namespace kl {

constexpr int kMaxSplits = 1024;

// The fixed scratch of keyless_decode_noalloc: its size, and its device address
// on the current device (looked up once per device, then cached).
constexpr size_t kScratchBytes = size_t(16) << 20;
hipError_t scratch_address(void** out);

// Raise a kernel's dynamic-LDS limit to `bytes`, once per device (devices
// 0..31 are remembered in `done`; others set it on every call).
inline hipError_t set_max_lds(const void* fn, int bytes, std::atomic<uint32_t>& done) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint32_t bit = (dev >= 0 && dev < 32) ? (1u << dev) : 0u;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
  return e;
}

struct DecodeParams {
  const void* q;          // [B, H, D]
  void* vdata;            // value cache data (written only by a fused append)
  const void* kdata;      // key cache data (standard decode) or nullptr
  const int32_t* table;   // paged block table or nullptr
  const int32_t* lengths; // [B]: rows to decode, or rows before the step when vnew is set
  const void* vnew;       // [B, G, D] the step's new value rows, or nullptr. When set, row
                          // lengths[b] of each sequence is the new row: it is appended to the
                          // cache (dropped past the capacity) and the decode covers
                          // lengths[b] + 1 rows, taking the new row from vnew
  void* out;              // [B, H, D]
  float* part;            // split partials: [B * H, S, D + 2] (split mode, S > 1) or
                          // [B * G + nwg, R, D + 2] (balanced mode)
  int* plan;              // balanced mode: [total tiles, tiles per workgroup, prefix[B + 1]]
  int B, H, G, D, R;
  kl_dtype dtype;
  bool paged;
  int L_max;              // contiguous capacity
  int block_shift;        // log2(block_size), paged
  int num_blocks, max_blocks;
  int chunk;              // rows per split (multiple of 64)
  int S;                  // splits per sequence (at most kMaxSplits)
  bool balanced;          // balanced mode: nwg workgroups share the tiles of all pairs evenly
  int nwg;                // workgroups in balanced mode (at most kMaxSplits)
  float scale_log2;       // scale * log2(e)
  hipEvent_t ev_start;    // optional: recorded around the split kernel
  hipEvent_t ev_stop;
};

hipError_t launch_decode(const DecodeParams& p, hipStream_t stream);

struct AppendParams {
  void* data;
  const void* values;     // [B, T, G, D]
  const int32_t* lengths_before;
  const int32_t* table;
  int B, T, G, D;
  kl_dtype dtype;
  bool paged;
  int L_max, block_shift, num_blocks, max_blocks;
};

hipError_t launch_append(const AppendParams& p, hipStream_t stream);

// Decode-step projections against packed weights Wp [N, K] (N = (H + G) D):
// out[b][n] = sum_k x[b][k] Wp[n][k], columns below NQ = H D to q_out, the rest
// to v_out and/or appended to the value cache at lengths_before[b]. bf16.
struct ProjectParams {
  const uint16_t* x;   // [B, K], row stride ldx
  const uint16_t* Wp;  // [N, K]
  uint16_t* q_out;     // [B, NQ], row stride ldq
  uint16_t* v_out;     // [B, N - NQ], row stride ldv, or nullptr
  uint16_t* cache;     // value cache data, or nullptr
  const int32_t* table;
  const int32_t* lengths_before;
  int B, K, N, NQ, G, D;
  long ldx, ldq, ldv;
  bool paged;
  int L_max, block_shift, num_blocks, max_blocks;
};

bool project_supported(int K);
hipError_t launch_project(const ProjectParams& p, hipStream_t stream);

// C[b] (M x N) = A[b] (M x K) * B[b] (K x N), row-major with leading
// dimensions, fp32 accumulation; batched by pointer strides. Generic tiled
// kernel for the small products (routing fold, fp32 prefill projections).
// C (M x N) = A (M x K) B (K x N) [+ C], fp32 arithmetic. Element (m, k) of A
// is at m lda + k a_cs, element (k, n) of B at k ldb + n b_cs (a_cs, b_cs of 0
// mean 1), so transposed operands are a choice of strides.
struct GemmParams {
  const void* A; const void* Bm; void* C;
  int M, N, K;
  long lda, ldb, ldc;
  long strideA, strideB, strideC;  // elements between batch items
  int batch;
  kl_dtype dtype;
  long a_cs, b_cs;
  int accumulate;                  // nonzero: C += A B
};

hipError_t launch_gemm_simple(const GemmParams& p, hipStream_t stream);

// bf16 MFMA GEMM: C (M x N) = A0 W0^T + A1 W1^T with A0 [M, K0], W0 [N, K0],
// A1 [M, K1], W1 [N, K1] (K contiguous in all four; K1 = 0 drops the second
// term). Columns < n_split go to C0, the rest to C1, bf16. Operand pointers
// must be 16-byte aligned.
struct GemmBf16Args {
  const void* A0;
  long lda0;
  const void* W0;
  long ldw0;
  int K0;
  const void* A1;
  long lda1;
  const void* W1;
  long ldw1;
  int K1;
  int M, N, n_split;
  void* C0;
  long ldc0;
  void* C1;
  long ldc1;
  // Batched (one term only): item (b, z) reads A0 + b sA0 + z zA0,
  // W0 + b sW0 + z zW0 and writes C0 + b sC0 + z zC0 (C1 likewise with sC1),
  // element strides; b < batch, z < zbatch.
  int batch;
  long sA0, sW0, sC0, sC1;
  int zbatch;
  long zA0, zW0, zC0;
  int c_f32;  // nonzero: C0, C1 are fp32 (one-term products)
};
// out[i] = bf16(sum over s < S of part[s n + i]) for i < n.
hipError_t launch_sum_partials_bf16(const float* part, int S, size_t n, void* out,
                                    hipStream_t stream);
// nullptr when the bf16 GEMM handles the shape, else the reason it does not.
const char* gemm_bf16_unsupported(const GemmBf16Args& a);
hipError_t launch_gemm_bf16(const GemmBf16Args& a, hipStream_t stream);
// The projection form: C = A (M x K, row-major) * Wp^T with Wp [N, K].
const char* gemm_bf16_unsupported(int M, int N, int K, long lda, long ldc0, long ldc1);
hipError_t launch_gemm_bf16_packed(const void* A, int M, int K, long lda, const void* Wp, int N,
                                   int n_split, void* C0, long ldc0, void* C1, long ldc1,
                                   hipStream_t stream);

// dst[c][r] = src[r][c] for r < rows, c < cols (bf16); dst columns r in
// [rows, rows_pad) are written as zeros. Row strides in elements; `batch`
// matrices s_src and s_dst elements apart.
hipError_t launch_transpose_bf16(const void* src, long ld_src, int rows, int cols, void* dst,
                                 long ld_dst, int rows_pad, hipStream_t stream, int batch = 1,
                                 long s_src = 0, long s_dst = 0);

// Packed projection weights: rows [0, H d) = (W^Q W^R per head)^T (or W^Q^T
// when W_R is null), rows [H d, (H+G) d) = W^V^T; each row has d_model entries.
struct PackParams {
  const void* W_Q;
  const void* W_R;
  const void* W_V;
  void* packed;
  int d_model, H, G, d_head, N;
};
hipError_t launch_pack_weights(const PackParams& p, hipStream_t stream);

struct AttnParams {
  const void* q;   // routed queries, [B, N, H, D] with row stride q_stride (elements per token)
  const void* v;   // values, [B, Nk, G, D] with row stride v_stride
  void* out;       // [B, N, H, D]
  long q_stride, v_stride, o_stride;
  int B, N, H, G, D;
  int Nk;          // value rows per sequence: N for self-attention, N_b for cross-attention
  int causal;      // only with Nk == N
  float* lse;      // [B, H, N] natural-log log-sum-exp of each row's scaled scores, or null
  float* out_f32;  // [B, N, H, D] the output before rounding to the dtype, or null
  float scale_log2;
  kl_dtype dtype;
};

// Latent cache products (Eq. 15): absorb y = x W_post_h^T (d_k -> r) or expand
// y = x W_post_h (r -> d_k) for every (sequence, head); r and d_k are 64 or 128.
struct LatentParams {
  const void* x;   // [B, H, n_in]
  const void* W;   // [H, r, d_k]
  void* y;         // [B, H, n_out]
  int B, H, r, dk;
  int absorb;
  kl_dtype dtype;
};
hipError_t launch_latent_product(const LatentParams& p, hipStream_t stream);

// Backward of the keyless self-attention (Section 2.3): dQ~ and dV from dO,
// the forward's output and log-sum-exp. q [B, N, H, D] (q_stride), v [B, N, G,
// D] (v_stride), out and dout [B, N, H, D] (o_stride), lse and Dd [B, H, N]
// fp32 (Dd is scratch: rowsum(dout * out)), dq [B, N, H, D] (dq_stride),
// dv [B, N, G, D] (dv_stride).
struct BwdParams {
  const void* q;
  const void* v;
  const void* out;
  const void* dout;
  const float* lse;
  const float* out_f32;  // [B, N, H, D] the forward's fp32 output, or null (then Dd is formed
                         // from P and dP in a first sweep of the dQ~ kernel)
  float* Dd;
  void* dq;
  void* dv;
  long q_stride, v_stride, o_stride, dq_stride, dv_stride;
  int B, N, H, G, D;
  int causal;
  float scale;       // tau
  float scale_log2;  // tau * log2(e)
  kl_dtype dtype;
};
bool attn_bwd_mfma_supported(const BwdParams& p);
hipError_t launch_attention_backward(const BwdParams& p, hipStream_t stream);

// bf16 MFMA flash-style keyless attention (d_head 64 or 128).
bool attn_bf16_supported(const AttnParams& p);
hipError_t launch_prefill_attention(const AttnParams& p, hipStream_t stream);
// fp32 (or fallback) VALU attention.
hipError_t launch_prefill_attention_simple(const AttnParams& p, hipStream_t stream);

// Measuring kernels (not part of the method): a streaming read of bytes (a
// multiple of 16, src 16-byte aligned) and a loop of matrix-core products,
// 4 waves x iters x 16 products of 16 x 16 x 32 per workgroup.
hipError_t launch_probe_read(const void* src, size_t bytes, unsigned* sink, int workgroups,
                             hipStream_t stream);
hipError_t launch_probe_mfma(float* sink, int iters, int workgroups, hipStream_t stream);

}  // namespace kl
