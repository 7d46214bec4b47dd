// bf16 MFMA GEMM for the prefill projections [Q~ | V] = X [W~^Q | W^V]
// (Eq. 2: no key projection). Two problems that share A run in one launch.
//
// C (M x N, bf16) = A (M x K, bf16, row-major) * B (K x N, bf16, row-major),
// fp32 accumulation in v_mfma_f32_16x16x32_bf16, one rounding to bf16 on store.
//
// Tile 256 x 256 x 64, 8 waves (2 x 4), each wave 128 x 64 of C. Both operands
// are staged in LDS K-major (64 k values of one row or column contiguous, rows
// padded by 16 bytes): A is copied as is; B arrives n-major from memory and is
// transposed in registers (4 x 8 blocks, v_perm) on its way into LDS. Global
// loads of tile k+1 are in flight while tile k is multiplied (two LDS buffers,
// 144 KiB). Workgroup ids are remapped so each XCD owns a band of 4 tile rows
// walked column-major, which keeps the A and B tiles of concurrently running
// workgroups in that XCD's L2.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int LDK = BK + 8;  // padded row length (elements) of an LDS tile
constexpr int kThreads = 512;

struct GemmBf16Params {
  const uint16_t* A;
  const uint16_t* B[2];
  uint16_t* C[2];
  int M, K;
  int N[2];
  long lda, ldb[2], ldc[2];
};

// Low halves of a and b -> (a.lo, b.lo); high halves -> (a.hi, b.hi).
__device__ __forceinline__ uint32_t lo_pair(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t hi_pair(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

__global__ __launch_bounds__(kThreads) void gemm_bf16_kernel(GemmBf16Params p) {
  const int prob = blockIdx.y;
  const int N = p.N[prob];
  const int tilesM = (p.M + BM - 1) / BM, tilesN = (N + BN - 1) / BN;
  const int ntiles = tilesM * tilesN;
  int wg = blockIdx.x;
  if (wg >= ntiles) return;
  // XCD-aware order: hardware places workgroup i on XCD i % 8.
  if (gridDim.x == (unsigned)ntiles && (ntiles & 7) == 0) wg = (wg & 7) * (ntiles >> 3) + (wg >> 3);
  constexpr int GM = 4;
  const int group = wg / (GM * tilesN);
  const int first_m = group * GM;
  const int gsize = min(tilesM - first_m, GM);
  const int in_group = wg % (GM * tilesN);
  const int tm = first_m + in_group % gsize;
  const int tn = in_group / gsize;
  const int m0 = tm * BM, n0 = tn * BN;

  const uint16_t* __restrict__ A = p.A;
  const uint16_t* __restrict__ Bm = p.B[prob];
  const long lda = p.lda, ldb = p.ldb[prob];

  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  uint16_t* As = smem;                    // [2][BM][LDK]
  uint16_t* Bs = smem + 2 * BM * LDK;     // [2][BN][LDK]

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int wm = wave >> 2, wn = wave & 3;

  // Global -> register staging assignments.
  const int a_chunk = t & 7, a_row = t >> 3;          // rows a_row + 64 i, 16 B chunk a_chunk
  const int b_nchunk = t & 31, b_kgroup = t >> 5;     // 4 k rows x 8 n columns
  u32x4 ra[4];
  u32x4 rb[4];

  auto load_global = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = m0 + a_row + 64 * i;
      const int rr = min(row, p.M - 1);
      ra[i] = *reinterpret_cast<const u32x4*>(A + (size_t)rr * lda + k0 + a_chunk * 8);
      if (row >= p.M) ra[i] = u32x4{0u, 0u, 0u, 0u};
    }
    const int col = n0 + b_nchunk * 8;
    const int cc = min(col, N - 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = k0 + b_kgroup * 4 + i;
      rb[i] = *reinterpret_cast<const u32x4*>(Bm + (size_t)k * ldb + cc);
      if (col >= N) rb[i] = u32x4{0u, 0u, 0u, 0u};
    }
  };

  auto store_lds = [&](int buf) {
    uint16_t* as = As + buf * BM * LDK;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<u32x4*>(as + (a_row + 64 * i) * LDK + a_chunk * 8) = ra[i];
    // Transpose the 4 (k) x 8 (n) block: column n gets its 4 k values (8 bytes).
    uint16_t* bs = Bs + buf * BN * LDK;
    uint32_t w01[8], w23[8];  // (k0,k1) and (k2,k3) pairs per n
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t a0 = rb[0][j], a1 = rb[1][j], a2 = rb[2][j], a3 = rb[3][j];
      w01[2 * j] = lo_pair(a0, a1);
      w01[2 * j + 1] = hi_pair(a0, a1);
      w23[2 * j] = lo_pair(a2, a3);
      w23[2 * j + 1] = hi_pair(a2, a3);
    }
#pragma unroll
    for (int n = 0; n < 8; ++n)
      *reinterpret_cast<u32x2*>(bs + (b_nchunk * 8 + n) * LDK + b_kgroup * 4) = u32x2{w01[n], w23[n]};
  };

  f32x4_t acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = p.K / BK;
  load_global(0);
  store_lds(0);
  __syncthreads();
  const int fr = lane & 15;          // fragment row (A) or column (B)
  const int fk = (lane >> 4) * 8;    // fragment k offset
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_global((kt + 1) * BK);
    const uint16_t* as = As + buf * BM * LDK + (wm * 128 + fr) * LDK + fk;
    const uint16_t* bs = Bs + buf * BN * LDK + (wn * 64 + fr) * LDK + fk;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8_t af[8], bf[4];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(as + i * 16 * LDK + ks * 32);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bf[j] = *reinterpret_cast<const bf16x8_t*>(bs + j * 16 * LDK + ks * 32);
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_lds(buf ^ 1);
    __syncthreads();
  }

  uint16_t* __restrict__ C = p.C[prob];
  const long ldc = p.ldc[prob];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + wn * 64 + j * 16 + fr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * 128 + i * 16 + (lane >> 4) * 4 + r;
        if (row < p.M && col < N)
          C[(size_t)row * ldc + col] = __builtin_bit_cast(uint16_t, (__bf16)acc[i][j][r]);
      }
    }
  }
}

}  // namespace

size_t gemm_bf16_lds_bytes() { return (size_t)2 * (BM + BN) * LDK * sizeof(uint16_t); }

// Validates shapes the kernel supports: K a multiple of 64, N and leading
// dimensions multiples of 8, N >= 8.
bool gemm_bf16_supported(int M, int N, int K, long lda, long ldb, long ldc) {
  return M > 0 && N >= 8 && K >= BK && K % BK == 0 && N % 8 == 0 && lda % 8 == 0 &&
         ldb % 8 == 0 && ldc % 8 == 0;
}

hipError_t launch_gemm_bf16_pair(const void* A, int M, int K, long lda, const void* B0,
                                 void* C0, int N0, long ldb0, long ldc0, const void* B1, void* C1,
                                 int N1, long ldb1, long ldc1, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_bf16_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)gemm_bf16_lds_bytes());
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  GemmBf16Params p{};
  p.A = static_cast<const uint16_t*>(A);
  p.M = M;
  p.K = K;
  p.lda = lda;
  p.B[0] = static_cast<const uint16_t*>(B0);
  p.C[0] = static_cast<uint16_t*>(C0);
  p.N[0] = N0;
  p.ldb[0] = ldb0;
  p.ldc[0] = ldc0;
  const int nprob = B1 ? 2 : 1;
  p.B[1] = static_cast<const uint16_t*>(B1 ? B1 : B0);
  p.C[1] = static_cast<uint16_t*>(B1 ? C1 : C0);
  p.N[1] = B1 ? N1 : N0;
  p.ldb[1] = B1 ? ldb1 : ldb0;
  p.ldc[1] = B1 ? ldc1 : ldc0;
  const int tilesM = (M + BM - 1) / BM;
  const int t0 = tilesM * ((p.N[0] + BN - 1) / BN), t1 = tilesM * ((p.N[1] + BN - 1) / BN);
  dim3 grid(t0 > t1 ? t0 : t1, nprob);
  hipLaunchKernelGGL(gemm_bf16_kernel, grid, dim3(kThreads), gemm_bf16_lds_bytes(), st, p);
  return hipGetLastError();
}

}  // namespace kl
