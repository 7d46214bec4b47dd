// One-time weight preparation before inference: the Section 2.1 fold
// W~^Q_h = W^Q_h W^R_h (done once, as Section 5.5 notes for the measured
// decode) and the packing of [W~^Q | W^V] into the operand layout of the
// projection GEMM and of the decode-step projection:
//   Wp [(H + G) d, d_model], row n = output column n, d_model contiguous;
//   rows h d + j (query head h):   Wp[h d + j][k] = sum_i W^Q[k][h d + i] W^R_h[i][j]
//                                  (W^Q[k][h d + j] itself without a routing matrix)
//   rows H d + n (value groups):   Wp[H d + n][k] = W^V[k][n]
//
// A workgroup (4 waves) owns one column block of d output rows (one query head
// or one value group) over KR consecutive k. The fold is a matrix-core product
// per 16-row block of k, D[k][j] = sum_i W^Q[k][h d + i] W^R_h[i][j] with
// v_mfma_f32_16x16x32_bf16: A = 16 rows of W^Q read straight from memory (16
// bytes per lane, the head's d columns of a row are contiguous), B = W^R_h,
// staged once per workgroup transposed in LDS so that a B fragment is one
// 16-byte LDS read; fp32 accumulation and one rounding to bf16. The value rows
// (and the query rows when there is no routing matrix) are a plain transpose,
// bit-exact. Either way the block is assembled in an LDS tile [n][k] and leaves
// it row by row with 16-byte stores, so both the reads and the writes of
// memory are whole 16-byte chunks of rows.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) uint16_t lds_u16;

constexpr int KR = 128;           // k (d_model rows) per workgroup
constexpr int kThreads = 256;     // 4 waves, each KR / 4 rows of k
constexpr int OROW = KR * 2 + 16; // bytes per row of the output tile [n][k] (padded)

template <int D>
struct PackTile {
  static constexpr int RROW = D * 2 + 16;  // bytes per row of the transposed W^R_h tile [j][i]
  static constexpr int OUT = D * OROW;     // output tile bytes
  static constexpr int RT = D * RROW;      // W^R_h tile bytes
};

__device__ __forceinline__ uint16_t half_of(const u32x4& v, int e) {
  return (uint16_t)((v[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
}

template <int D, bool FOLD>
__global__ __launch_bounds__(kThreads) void pack_weights_kernel(PackParams p) {
  using T = PackTile<D>;
  constexpr int CH = D / 8;  // 16-byte chunks of a row's d columns
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  lds_u8* const otile = (lds_u8*)smem;
  lds_u8* const rtile = (lds_u8*)smem + T::OUT;

  const int cb = blockIdx.x;  // query head cb (cb < H) or value group cb - H
  const int k0 = blockIdx.y * KR;
  const int krows = min(KR, p.d_model - k0);
  const int t = threadIdx.x;
  const bool query = cb < p.H;
  const uint16_t* src;
  long ld;
  if (query) {
    src = static_cast<const uint16_t*>(p.W_Q) + (size_t)cb * D;
    ld = (long)p.H * D;
  } else {
    src = static_cast<const uint16_t*>(p.W_V) + (size_t)(cb - p.H) * D;
    ld = (long)p.G * D;
  }

  if (FOLD && query) {
    // rtile[j][i] = W^R_h[i][j]; consecutive lanes take consecutive i, so the
    // 2-byte LDS writes of one instruction fall in distinct banks.
    const uint16_t* R = static_cast<const uint16_t*>(p.W_R) + (size_t)cb * D * D;
    for (int c = t; c < D * CH; c += kThreads) {
      const int i = c % D, jc = c / D;
      const u32x4 v = *reinterpret_cast<const u32x4*>(R + (size_t)i * D + jc * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        *(lds_u16*)(rtile + (jc * 8 + e) * T::RROW + i * 2) = half_of(v, e);
    }
    __syncthreads();
    const int lane = t & 63, wave = t >> 6;
    const int fr = lane & 15, grp = lane >> 4;
    constexpr int KS = D / 32, DB = D / 16;
#pragma unroll
    for (int kb = 0; kb < KR / 64; ++kb) {
      const int kr = wave * (KR / 4) + kb * 16;  // first tile row of this 16-row block
      const int k = k0 + kr + fr;                // lane's A row
      bf16x8_t a[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        u32x4 v{0u, 0u, 0u, 0u};
        if (kr + fr < krows) v = *reinterpret_cast<const u32x4*>(src + (size_t)k * ld + ks * 32 + grp * 8);
        a[ks] = __builtin_bit_cast(bf16x8_t, v);
      }
#pragma unroll
      for (int jb = 0; jb < DB; ++jb) {
        f32x4_t acc{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8_t b = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
              rtile + (jb * 16 + fr) * T::RROW + (ks * 32 + grp * 8) * 2);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], b, acc, 0, 0, 0);
        }
        // Lane holds D[kr + 4 grp + r][16 jb + fr], r = 0..3: four consecutive k of row n.
        typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 w{pack_bf16(acc[0], acc[1]), pack_bf16(acc[2], acc[3])};
        *(__attribute__((address_space(3))) u32x2*)(otile + (jb * 16 + fr) * OROW + (kr + grp * 4) * 2) = w;
      }
    }
  } else {
    // otile[n][k] = source[k][n]; consecutive lanes take consecutive k.
    for (int c = t; c < KR * CH; c += kThreads) {
      const int kr = c % KR, nc = c / KR;
      u32x4 v{0u, 0u, 0u, 0u};
      if (kr < krows) v = *reinterpret_cast<const u32x4*>(src + (size_t)(k0 + kr) * ld + nc * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) *(lds_u16*)(otile + (nc * 8 + e) * OROW + kr * 2) = half_of(v, e);
    }
  }
  __syncthreads();

  // Rows of the tile to Wp[cb d + n][k0 ..]: 16 bytes per lane, whole rows per
  // group of KR / 8 lanes; a ragged end of d_model (or rows that are not
  // 16-byte aligned) is stored element by element.
  uint16_t* out = static_cast<uint16_t*>(p.packed);
  constexpr int OCH = KR / 8;
  const bool vec = (p.d_model & 7) == 0;
  for (int c = t; c < D * OCH; c += kThreads) {
    const int n = c / OCH, kk = (c % OCH) * 8;
    if (kk >= krows) continue;
    uint16_t* dst = out + (size_t)(cb * D + n) * p.d_model + k0 + kk;
    const u32x4 v = *(__attribute__((address_space(3))) u32x4*)(otile + n * OROW + kk * 2);
    if (vec && kk + 8 <= krows) {
      *reinterpret_cast<u32x4*>(dst) = v;
    } else {
      for (int e = 0; e < 8 && kk + e < krows; ++e) dst[e] = half_of(v, e);
    }
  }
}

template <int D, bool FOLD>
hipError_t launch_pack(const PackParams& p, hipStream_t st) {
  using T = PackTile<D>;
  const int lds = T::OUT + (FOLD ? T::RT : 0);
  static std::atomic<uint32_t> attr_done{0};
  hipError_t e = set_max_lds((const void*)pack_weights_kernel<D, FOLD>, lds, attr_done);
  if (e != hipSuccess) return e;
  dim3 grid(p.H + p.G, (p.d_model + KR - 1) / KR);
  hipLaunchKernelGGL((pack_weights_kernel<D, FOLD>), grid, dim3(kThreads), lds, st, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pack_weights(const PackParams& p, hipStream_t st) {
  if (p.d_model <= 0 || p.H <= 0 || p.G <= 0) return hipErrorInvalidValue;
  if (p.d_head == 128) return p.W_R ? launch_pack<128, true>(p, st) : launch_pack<128, false>(p, st);
  if (p.d_head == 64) return p.W_R ? launch_pack<64, true>(p, st) : launch_pack<64, false>(p, st);
  return hipErrorInvalidValue;
}

}  // namespace kl
