// bf16 MFMA GEMM for the prefill projections [Q~ | V] = X [W~^Q | W^V]
// (Eq. 2: no key projection), against weights packed once before inference,
// and for the large products of the backward pass through the projections.
//
// C (M x N) = A0 W0^T + A1 W1^T, where A0 [M, K0] and W0 [N, K0] (row n =
// output column n) are both K-major, the layout the MFMA fragments want; the
// optional second term (K1 > 0) continues the same k loop on another pair of
// operands. For the projections A0 = X, W0 = the packed weights and K1 = 0.
// Columns below n_split go to C0 (the routed queries), the rest to C1 (the
// values). fp32 accumulation in v_mfma_f32_16x16x32_bf16, one rounding to
// bf16 on store.
//
// Tile 256 x 256 x 64, 16 waves (4 x 4), each wave 64 x 64 of C (64 fp32
// accumulators per lane, four waves per SIMD: while some waves restart a k-tile
// with their LDS reads after the barrier, others keep the matrix pipe busy). Each operand tile is 256 rows of
// 128 bytes in LDS with the 16-byte chunks of row r XOR-swizzled by
// (r >> 1) & 7, so the fragment reads (16 rows per access) are free of bank
// conflicts. Tiles move from memory straight into LDS (global_load_lds, 16
// bytes per lane, no register staging); the swizzle is applied to the global
// addresses. Two LDS stages (128 KiB): the next tile is in flight while the
// current one is multiplied.
// Workgroup ids are remapped so each XCD owns a band of tile rows walked
// column-major, which keeps concurrently running tiles in that XCD's L2.

#include <type_traits>

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((address_space(3))) unsigned char lds_u8;

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 1024;
constexpr int TILE_BYTES = 256 * BK * 2;  // one operand tile, 32 KiB
static_assert(BK == 64, "the fragment schedule assumes two 32-wide k-steps per tile");

struct GemmParams2 {
  const uint16_t* A0;  // [M, K0], row stride lda0 (elements)
  const uint16_t* W0;  // [N, K0], row stride ldw0
  const uint16_t* A1;  // [M, K1], row stride lda1 (K1 = 0: no second term)
  const uint16_t* W1;  // [N, K1], row stride ldw1
  void* C0;            // columns [0, n_split): bf16, or fp32 for the F32 form
  void* C1;            // columns [n_split, N)
  int M, N, K0, K1, n_split;
  long lda0, ldw0, lda1, ldw1;
  long ldc0, ldc1;
  long sA0, sW0, sC0, sC1;  // element strides between batch items (blockIdx.y)
  long zA0, zW0, zC0;       // and along blockIdx.z (a second batch index)
};

// Byte offset of (row, 16-byte chunk) inside a swizzled operand tile.
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * (BK * 2) + ((chunk ^ ((row >> 1) & 7)) << 4);
}

// Four waves per SIMD (the 128 KiB of LDS allow one workgroup per CU): the
// register budget is 128, the accumulators and one k-step's fragments.
// TWO: the second term is present (one more pair of copy offsets per lane and
// a uniform choice per k-tile; the projections take the plain form). F32: the
// outputs are stored in fp32 (partial products of a split contraction).
template <bool TWO, bool F32>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemm_bf16_kernel(GemmParams2 p) {
  using CT = std::conditional_t<F32, float, uint16_t>;
  const int tilesM = (p.M + BM - 1) / BM, tilesN = (p.N + BN - 1) / BN;
  const int ntiles = tilesM * tilesN;
  CT* C0 = static_cast<CT*>(p.C0);
  CT* C1 = static_cast<CT*>(p.C1);
  if (blockIdx.y > 0 || blockIdx.z > 0) {  // batch item: the first term's operands and the outputs move
    p.A0 += (size_t)blockIdx.y * p.sA0 + (size_t)blockIdx.z * p.zA0;
    p.W0 += (size_t)blockIdx.y * p.sW0 + (size_t)blockIdx.z * p.zW0;
    C0 += (size_t)blockIdx.y * p.sC0 + (size_t)blockIdx.z * p.zC0;
    C1 += (size_t)blockIdx.y * p.sC1 + (size_t)blockIdx.z * p.zC0;
  }
  int wg = blockIdx.x;
  // XCD-aware order: hardware places workgroup i on XCD i % 8.
  if ((ntiles & 7) == 0) wg = (wg & 7) * (ntiles >> 3) + (wg >> 3);
  constexpr int GM = 4;
  const int group = wg / (GM * tilesN);
  const int first_m = group * GM;
  const int gsize = min(tilesM - first_m, GM);
  const int in_group = wg % (GM * tilesN);
  const int m0 = (first_m + in_group % gsize) * BM;
  const int n0 = (in_group / gsize) * BN;

  // Two pipeline stages, each an A tile and a W tile: [stage][A | W].
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 2, wn = wave & 3;  // wave tile: rows 64 wm.., columns 64 wn..

  // Direct-to-LDS copies: one wave instruction fills 8 rows (1 KiB) of a tile,
  // lane L landing at byte 16 L, i.e. row L / 8, physical chunk L % 8, which
  // holds logical chunk (L % 8) ^ ((row >> 1) & 7). Each wave fills 2 row groups
  // of each operand. Rows past the end are clamped: they only feed output rows
  // or columns that are never stored. Per-lane byte offsets for each term.
  constexpr int NT = TWO ? 2 : 1;
  uint32_t offA[NT][2], offW[NT][2];  // [term][row group]
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (i * 16 + wave) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((r >> 1) & 7);
    const int ra = min(m0 + r, p.M - 1), rw = min(n0 + r, p.N - 1);
    offA[0][i] = (uint32_t)(((size_t)ra * p.lda0 + lc * 8) * 2);
    offW[0][i] = (uint32_t)(((size_t)rw * p.ldw0 + lc * 8) * 2);
    if constexpr (TWO) {
      offA[NT - 1][i] = (uint32_t)(((size_t)ra * p.lda1 + lc * 8) * 2);
      offW[NT - 1][i] = (uint32_t)(((size_t)rw * p.ldw1 + lc * 8) * 2);
    }
  }
  const int nk0 = p.K0 / BK;  // k-tiles of the first term
  // Copies of k-tile kt (of the concatenated k range) into one stage.
  auto issue = [&](lds_u8* sa, lds_u8* sw, int kt) {
    const bool second = TWO && kt >= nk0;  // uniform
    const int k0 = (second ? kt - nk0 : kt) * BK;
    const unsigned char* ga = reinterpret_cast<const unsigned char*>(second ? p.A1 : p.A0) + (size_t)k0 * 2;
    const unsigned char* gw = reinterpret_cast<const unsigned char*>(second ? p.W1 : p.W0) + (size_t)k0 * 2;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t grp_off = (uint32_t)((i * 16 + wave) * 1024);
      copy_to_lds(ga, second ? offA[NT - 1][i] : offA[0][i], (uint32_t)(uintptr_t)sa + grp_off);
      copy_to_lds(gw, second ? offW[NT - 1][i] : offW[0][i], (uint32_t)(uintptr_t)sw + grp_off);
    }
  };

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, grp = lane >> 4;
  // Per 32-wide k-step: the wave's 4 A and 4 W fragments, then its 16 products
  // (one fragment set; the other three waves on the SIMD cover the read latency).
  auto compute = [&](const lds_u8* a, const lds_u8* w) {
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      const int chunk = ks * 4 + grp;
      bf16x8_t af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
            a + swz(wm * 64 + i * 16 + fr, chunk));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bf[j] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
            w + swz(wn * 64 + j * 16 + fr, chunk));
      // W as the A operand: the result block is C^T, so a lane holds four
      // consecutive output columns of one row (one 8-byte store in bf16).
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bf[j], af[i], acc[i][j], 0, 0, 0);
    }
  };

  lds_u8* const base = (lds_u8*)smem;
  auto stageA = [&](int st) { return base + st * 2 * TILE_BYTES; };
  auto stageW = [&](int st) { return base + st * 2 * TILE_BYTES + TILE_BYTES; };
  const int nk = TWO ? nk0 + p.K1 / BK : nk0;
  issue(stageA(0), stageW(0), 0);
  // One barrier per k-tile. Before it, each wave waits for its copies of tile
  // kt (the only ones in flight) and for its own LDS reads of tile kt - 1 (the
  // barrier does not wait for those); after it, both hold for every wave, so
  // the copies of tile kt + 1 may refill the stage of tile kt - 1 while tile kt
  // is multiplied.
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    KL_WAIT_VMCNT(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __syncthreads();
    if (kt + 1 < nk) issue(stageA(cur ^ 1), stageW(cur ^ 1), kt + 1);
    compute(stageA(cur), stageW(cur));
  }

  // Lane holds C[row 16 i + fr][col 16 j + 4 grp + r] of the wave's 64 x 64 block:
  // four consecutive columns, stored as one 8-byte (bf16) or 16-byte (fp32)
  // store when they lie on one side of n_split, inside N, and the outputs' row
  // strides and bases keep them aligned (uniform); otherwise element by element.
  // A tile whose rows all exist stores without a per-row check.
  constexpr int VB = 4 * (int)sizeof(CT);  // bytes of four outputs
  const bool vec = p.ldc0 % 4 == 0 && p.ldc1 % 4 == 0 && p.n_split % 4 == 0 &&
                   reinterpret_cast<uintptr_t>(C0) % VB == 0 &&
                   reinterpret_cast<uintptr_t>(C1) % VB == 0;
  auto store = [&](auto check_rows) {
    constexpr bool CHECK = decltype(check_rows)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = m0 + wm * 64 + i * 16 + fr;
      if (CHECK && row >= p.M) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + wn * 64 + j * 16 + grp * 4;
        if (vec && col + 4 <= p.N && (col + 4 <= p.n_split || col >= p.n_split)) {
          CT* dst = col < p.n_split ? C0 + (size_t)row * p.ldc0 + col
                                    : C1 + (size_t)row * p.ldc1 + (col - p.n_split);
          if constexpr (F32) {
            *reinterpret_cast<f32x4_t*>(dst) = acc[i][j];
          } else {
            typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
            const bf16x4_t v = {(__bf16)acc[i][j][0], (__bf16)acc[i][j][1], (__bf16)acc[i][j][2],
                                (__bf16)acc[i][j][3]};
            *reinterpret_cast<bf16x4_t*>(dst) = v;
          }
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int c = col + r;
            if (c >= p.N) continue;
            CT* dst = c < p.n_split ? C0 + (size_t)row * p.ldc0 + c
                                    : C1 + (size_t)row * p.ldc1 + (c - p.n_split);
            if constexpr (F32) *dst = acc[i][j][r];
            else *dst = __builtin_bit_cast(uint16_t, (__bf16)acc[i][j][r]);
          }
        }
      }
    }
  };
  if (m0 + BM <= p.M) store(std::false_type{});
  else store(std::true_type{});
}

}  // namespace

const char* gemm_bf16_unsupported(const GemmBf16Args& a) {
  if (a.M <= 0 || a.N <= 0) return "empty product";
  if (a.K0 < BK || a.K0 % BK != 0 || a.K1 < 0 || a.K1 % BK != 0)
    return "the contraction lengths must be multiples of 64 (the first one positive)";
  if (a.lda0 % 8 != 0 || a.lda0 < a.K0 || a.ldw0 % 8 != 0 || a.ldw0 < a.K0)
    return "operand row strides must be multiples of 8 and at least the contraction length";
  if (a.K1 > 0 && (a.lda1 % 8 != 0 || a.lda1 < a.K1 || a.ldw1 % 8 != 0 || a.ldw1 < a.K1))
    return "operand row strides must be multiples of 8 and at least the contraction length";
  if (a.ldc0 <= 0 || a.ldc1 <= 0) return "output row strides must be positive";
  if ((a.batch > 1 || a.zbatch > 1) &&
      (a.K1 > 0 || a.batch > 65535 || a.zbatch > 65535 || a.sA0 % 8 != 0 || a.sW0 % 8 != 0 ||
       a.zA0 % 8 != 0 || a.zW0 % 8 != 0))
    return "a batched product has one term, at most 65535 items per index, and 16-byte aligned items";
  if (a.c_f32 && a.K1 > 0) return "fp32 outputs are for one-term products";
  // Operand offsets are 32-bit byte offsets.
  const size_t lim = 1ull << 32;
  if ((size_t)a.M * a.lda0 * 2 >= lim || (size_t)a.N * a.ldw0 * 2 >= lim ||
      (a.K1 > 0 && ((size_t)a.M * a.lda1 * 2 >= lim || (size_t)a.N * a.ldw1 * 2 >= lim)))
    return "an operand exceeds 4 GiB (32-bit operand offsets)";
  return nullptr;
}

const char* gemm_bf16_unsupported(int M, int N, int K, long lda, long ldc0, long ldc1) {
  GemmBf16Args a{};
  a.M = M;
  a.N = N;
  a.K0 = K;
  a.lda0 = lda;
  a.ldw0 = K;
  a.ldc0 = ldc0;
  a.ldc1 = ldc1;
  const char* why = gemm_bf16_unsupported(a);
  if (why && (K < BK || K % BK != 0)) return "d_model must be a positive multiple of 64 for bf16";
  if (why && (lda % 8 != 0 || lda < K))
    return "the row stride of x must be a multiple of 8 and >= d_model";
  return why;
}

constexpr size_t kGemmLds = 4 * TILE_BYTES;

hipError_t launch_gemm_bf16(const GemmBf16Args& a, hipStream_t st) {
  static std::atomic<uint32_t> attr_one{0}, attr_two{0}, attr_f32{0};
  const void* kern = a.K1 > 0 ? (const void*)gemm_bf16_kernel<true, false>
                   : a.c_f32  ? (const void*)gemm_bf16_kernel<false, true>
                              : (const void*)gemm_bf16_kernel<false, false>;
  {
    hipError_t e = set_max_lds(kern, (int)kGemmLds,
                               a.K1 > 0 ? attr_two : (a.c_f32 ? attr_f32 : attr_one));
    if (e != hipSuccess) return e;
  }
  GemmParams2 p{};
  p.A0 = static_cast<const uint16_t*>(a.A0);
  p.W0 = static_cast<const uint16_t*>(a.W0);
  p.A1 = static_cast<const uint16_t*>(a.K1 > 0 ? a.A1 : a.A0);
  p.W1 = static_cast<const uint16_t*>(a.K1 > 0 ? a.W1 : a.W0);
  p.C0 = a.C0;
  p.C1 = a.C1;
  p.M = a.M;
  p.N = a.N;
  p.K0 = a.K0;
  p.K1 = a.K1;
  p.n_split = a.n_split;
  p.lda0 = a.lda0;
  p.ldw0 = a.ldw0;
  p.lda1 = a.K1 > 0 ? a.lda1 : a.lda0;
  p.ldw1 = a.K1 > 0 ? a.ldw1 : a.ldw0;
  p.ldc0 = a.ldc0;
  p.ldc1 = a.ldc1;
  p.sA0 = a.sA0;
  p.sW0 = a.sW0;
  p.sC0 = a.sC0;
  p.sC1 = a.sC1;
  p.zA0 = a.zA0;
  p.zW0 = a.zW0;
  p.zC0 = a.zC0;
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  const dim3 grid(tiles, a.batch > 1 ? a.batch : 1, a.zbatch > 1 ? a.zbatch : 1);
  if (a.K1 > 0)
    hipLaunchKernelGGL((gemm_bf16_kernel<true, false>), grid, dim3(kThreads), kGemmLds, st, p);
  else if (a.c_f32)
    hipLaunchKernelGGL((gemm_bf16_kernel<false, true>), grid, dim3(kThreads), kGemmLds, st, p);
  else
    hipLaunchKernelGGL((gemm_bf16_kernel<false, false>), grid, dim3(kThreads), kGemmLds, st, p);
  return hipGetLastError();
}

namespace {

// out[i] = bf16(sum over s < S of part[s n + i]), in order of s.
__global__ __launch_bounds__(256) void sum_partials_kernel(const float* __restrict__ part, int S,
                                                           size_t n, uint16_t* __restrict__ out) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float acc = 0.f;
  for (int s = 0; s < S; ++s) acc += part[(size_t)s * n + i];
  out[i] = __builtin_bit_cast(uint16_t, (__bf16)acc);
}

}  // namespace

hipError_t launch_sum_partials_bf16(const float* part, int S, size_t n, void* out, hipStream_t st) {
  if (n == 0) return hipSuccess;
  if (S <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sum_partials_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, part,
                     S, n, static_cast<uint16_t*>(out));
  return hipGetLastError();
}

hipError_t launch_gemm_bf16_packed(const void* A, int M, int K, long lda, const void* Wp, int N,
                                   int n_split, void* C0, long ldc0, void* C1, long ldc1,
                                   hipStream_t st) {
  GemmBf16Args a{};
  a.A0 = A;
  a.lda0 = lda;
  a.W0 = Wp;
  a.ldw0 = K;
  a.K0 = K;
  a.M = M;
  a.N = N;
  a.n_split = n_split;
  a.C0 = C0;
  a.ldc0 = ldc0;
  a.C1 = C1;
  a.ldc1 = ldc1;
  return launch_gemm_bf16(a, st);
}

}  // namespace kl

