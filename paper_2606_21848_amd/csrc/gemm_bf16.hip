// bf16 MFMA GEMM for the prefill projections [Q~ | V] = X [W~^Q | W^V]
// (Eq. 2: no key projection), against weights packed once before inference.
//
// C (M x N) = A (M x K) * Wp^T, where A = X is row-major [M, K] and Wp is the
// packed weight [N, K] (row n = output column n, K contiguous): both operands
// are K-major, which is the layout the MFMA fragments want. Columns below
// n_split go to C0 (the routed queries), the rest to C1 (the values).
// fp32 accumulation in v_mfma_f32_16x16x32_bf16, one rounding to bf16 on store.
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
  const uint16_t* A;   // [M, K]
  const uint16_t* W;   // [N, K] packed
  uint16_t* C0;        // columns [0, n_split)
  uint16_t* C1;        // columns [n_split, N)
  int M, N, K, n_split;
  long lda;            // A row stride (elements)
  long ldc0, ldc1;
};

// Byte offset of (row, 16-byte chunk) inside a swizzled operand tile.
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * (BK * 2) + ((chunk ^ ((row >> 1) & 7)) << 4);
}

// Four waves per SIMD (the 128 KiB of LDS allow one workgroup per CU): the
// register budget is 128, the accumulators and one k-step's fragments.
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemm_bf16_kernel(GemmParams2 p) {
  const int tilesM = (p.M + BM - 1) / BM, tilesN = (p.N + BN - 1) / BN;
  const int ntiles = tilesM * tilesN;
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
  // or columns that are never stored.
  uint32_t offA[2], offW[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (i * 16 + wave) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((r >> 1) & 7);
    const int ra = min(m0 + r, p.M - 1), rw = min(n0 + r, p.N - 1);
    offA[i] = (uint32_t)(((size_t)ra * p.lda + lc * 8) * 2);
    offW[i] = (uint32_t)(((size_t)rw * p.K + lc * 8) * 2);
  }
  const unsigned char* gA = reinterpret_cast<const unsigned char*>(p.A);
  const unsigned char* gW = reinterpret_cast<const unsigned char*>(p.W);
  auto issue = [&](lds_u8* sa, lds_u8* sw, int k0) {
    const unsigned char* ga = gA + (size_t)k0 * 2;
    const unsigned char* gw = gW + (size_t)k0 * 2;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t grp_off = (uint32_t)((i * 16 + wave) * 1024);
      copy_to_lds(ga, offA[i], (uint32_t)(uintptr_t)sa + grp_off);
      copy_to_lds(gw, offW[i], (uint32_t)(uintptr_t)sw + grp_off);
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
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  };

  lds_u8* const base = (lds_u8*)smem;
  auto stageA = [&](int st) { return base + st * 2 * TILE_BYTES; };
  auto stageW = [&](int st) { return base + st * 2 * TILE_BYTES + TILE_BYTES; };
  const int nk = p.K / BK;
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
    if (kt + 1 < nk) issue(stageA(cur ^ 1), stageW(cur ^ 1), (kt + 1) * BK);
    compute(stageA(cur), stageW(cur));
  }

  // Lane holds C[row 16 i + 4 grp + r][col 16 j + fr] of the wave's 64 x 64 block.
  // A tile whose rows all exist stores without a per-element row check.
  auto store = [&](auto check_rows) {
    constexpr bool CHECK = decltype(check_rows)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + wn * 64 + j * 16 + fr;
      if (col >= p.N) continue;
      uint16_t* dst;
      long ldc;
      if (col < p.n_split) {
        dst = p.C0 + col;
        ldc = p.ldc0;
      } else {
        dst = p.C1 + (col - p.n_split);
        ldc = p.ldc1;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + wm * 64 + i * 16 + grp * 4 + r;
          if (!CHECK || row < p.M)
            dst[(size_t)row * ldc] = __builtin_bit_cast(uint16_t, (__bf16)acc[i][j][r]);
        }
    }
  };
  if (m0 + BM <= p.M) store(std::false_type{});
  else store(std::true_type{});
}

}  // namespace

const char* gemm_bf16_unsupported(int M, int N, int K, long lda, long ldc0, long ldc1) {
  if (M <= 0 || N <= 0) return "empty product";
  if (K < BK || K % BK != 0) return "d_model must be a positive multiple of 64 for bf16";
  if (lda % 8 != 0 || lda < K) return "the row stride of x must be a multiple of 8 and >= d_model";
  if (ldc0 <= 0 || ldc1 <= 0) return "output row strides must be positive";
  // Operand offsets are 32-bit byte offsets.
  if ((size_t)M * lda * 2 >= (1ull << 32) || (size_t)N * K * 2 >= (1ull << 32))
    return "x or the packed weights exceed 4 GiB (32-bit operand offsets)";
  return nullptr;
}

constexpr size_t kGemmLds = 4 * TILE_BYTES;

hipError_t launch_gemm_bf16_packed(const void* A, int M, int K, long lda, const void* Wp, int N,
                                   int n_split, void* C0, long ldc0, void* C1, long ldc1,
                                   hipStream_t st) {
  static std::atomic<uint32_t> attr_done{0};
  {
    hipError_t e = set_max_lds((const void*)gemm_bf16_kernel, (int)kGemmLds, attr_done);
    if (e != hipSuccess) return e;
  }
  GemmParams2 p{};
  p.A = static_cast<const uint16_t*>(A);
  p.W = static_cast<const uint16_t*>(Wp);
  p.C0 = static_cast<uint16_t*>(C0);
  p.C1 = static_cast<uint16_t*>(C1);
  p.M = M;
  p.N = N;
  p.K = K;
  p.n_split = n_split;
  p.lda = lda;
  p.ldc0 = ldc0;
  p.ldc1 = ldc1;
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  hipLaunchKernelGGL(gemm_bf16_kernel, dim3(tiles), dim3(kThreads), kGemmLds, st, p);
  return hipGetLastError();
}

}  // namespace kl

