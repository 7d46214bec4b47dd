// Causal (or full) keyless attention for the bf16 prefill (Eq. 2 with the score
// of Eq. 4): O_h = softmax(tau * Q~_h V_g^T) V_g, where the value tile is both
// the "key" of the score and the value of the weighted sum.
//
// A workgroup (4 waves) owns 128 query rows of one head; each wave owns 32 rows.
// The routed-query fragments stay in registers. For every 64-row value tile,
// read from memory once, two LDS copies are written: row-major (rows of d_head
// contiguous) and transposed (64 rows of one column contiguous, built in
// registers with v_perm). Then, with v_mfma_f32_16x16x32_bf16:
//   S^T = V Q~^T     A operand = value rows (row-major copy), B = routed queries
//   O^T += V^T P^T   A operand = value columns (transposed copy), B = P in bf16
// Computing S^T leaves each lane holding scores of a single query row, so the
// online softmax needs only two cross-lane steps per row, and the score
// registers become the B operand of the second product without a transpose
// (the MFMA reduction order over a 32-row step is free as long as both operands
// agree; here a lane group g covers rows 4g..4g+3 and 16+4g..16+4g+3).
// The next value tile is loaded from memory while the current one is used.
// Causal work grows with the query tile, so the last tiles are scheduled first.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int BQ = 128;   // query rows per workgroup
constexpr int BKV = 64;   // value rows per tile
constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t lo_pair(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t hi_pair(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 b2;
  b2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

template <int D>
struct AttnLds {
  static constexpr int VS_LD = D + 8;     // row-major copy: [BKV][D + 8]
  static constexpr int VT_LD = BKV + 8;   // transposed copy: [D][BKV + 8]
  static constexpr int VS = BKV * VS_LD;  // elements
  static constexpr int VT = D * VT_LD;
  static constexpr int BUF = VS + VT;
  static constexpr size_t BYTES = 2 * BUF * sizeof(uint16_t);
};

template <int D>
__global__ __launch_bounds__(kThreads) void attn_bf16_kernel(AttnParams p) {
  using L = AttnLds<D>;
  constexpr int KS = D / 32;       // MFMA k-steps over d_head for S^T
  constexpr int DB = D / 16;       // 16-wide column blocks of the output
  constexpr int DCH = D / 8;       // 16-byte chunks per value row
  constexpr int LOADERS = (BKV / 4) * DCH;  // threads that load a 4 x 8 block each

  const int ntq = (p.N + BQ - 1) / BQ;
  const int qt = p.causal ? (ntq - 1 - (int)blockIdx.x) : (int)blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (p.H / p.G);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int fr = lane & 15, grp = lane >> 4;
  const int q0 = qt * BQ + wave * 32;  // this wave's first query row

  const uint16_t* __restrict__ Q = reinterpret_cast<const uint16_t*>(p.q);
  const uint16_t* __restrict__ V = reinterpret_cast<const uint16_t*>(p.v);

  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];

  // Routed-query fragments (B operand of S^T): query row q0 + 16 qb + fr,
  // columns 32 ks + 8 grp .. + 7.
  bf16x8_t qf[2][KS];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int q = q0 + qb * 16 + fr;
    const int qq = min(q, p.N - 1);
    const uint16_t* src = Q + ((size_t)b * p.N + qq) * p.q_stride + (size_t)h * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 w = *reinterpret_cast<const u32x4*>(src + ks * 32);
      if (q >= p.N) w = u32x4{0u, 0u, 0u, 0u};
      qf[qb][ks] = __builtin_bit_cast(bf16x8_t, w);
    }
  }

  f32x4_t o[DB][2];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i][0] = o[i][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m[2] = {-INFINITY, -INFINITY};
  float lsum[2] = {0.f, 0.f};  // per-lane partial sums; reduced at the end

  // Value-tile loader: thread t < LOADERS moves a 4-row x 8-column block.
  const bool loader = t < LOADERS;
  const int ld_ch = t % DCH, ld_grp = t / DCH;
  u32x4 rv[4];
  const size_t vrow0 = (size_t)b * p.N;
  auto load_tile = [&](int j0) {
    if (!loader) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = j0 + ld_grp * 4 + i;
      const int rr = min(row, p.N - 1);
      rv[i] = *reinterpret_cast<const u32x4*>(V + (vrow0 + rr) * p.v_stride + (size_t)g * D + ld_ch * 8);
      if (row >= p.N) rv[i] = u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_tile = [&](int buf) {
    if (!loader) return;
    uint16_t* vs = smem + buf * L::BUF;
    uint16_t* vt = vs + L::VS;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<u32x4*>(vs + (ld_grp * 4 + i) * L::VS_LD + ld_ch * 8) = rv[i];
    uint32_t w01[8], w23[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      w01[2 * j] = lo_pair(rv[0][j], rv[1][j]);
      w01[2 * j + 1] = hi_pair(rv[0][j], rv[1][j]);
      w23[2 * j] = lo_pair(rv[2][j], rv[3][j]);
      w23[2 * j + 1] = hi_pair(rv[2][j], rv[3][j]);
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
      *reinterpret_cast<u32x2*>(vt + (ld_ch * 8 + c) * L::VT_LD + ld_grp * 4) = u32x2{w01[c], w23[c]};
  };

  // Value tiles this workgroup needs.
  const int last_row = p.causal ? min(qt * BQ + BQ, p.N) : p.N;
  const int ntiles = (last_row + BKV - 1) / BKV;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int jt = 0; jt < ntiles; ++jt) {
    const int buf = jt & 1;
    const int j0 = jt * BKV;
    if (jt + 1 < ntiles) load_tile(j0 + BKV);
    const uint16_t* vs = smem + buf * L::BUF;
    const uint16_t* vt = vs + L::VS;
    // Skip tiles entirely above the diagonal for this wave.
    const bool live = !p.causal || j0 <= q0 + 31;
    if (live) {
      // S^T[kv][q] for kv blocks kb (16 rows) and query blocks qb.
      f32x4_t s[4][2];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        s[kb][0] = s[kb][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(
              vs + (kb * 16 + fr) * L::VS_LD + ks * 32 + grp * 8);
          s[kb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[0][ks], s[kb][0], 0, 0, 0);
          s[kb][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[1][ks], s[kb][1], 0, 0, 0);
        }
      }
      // Lane holds scores of query q0 + 16 qb + fr against rows j0 + 16 kb + 4 grp + r.
      const bool need_mask = (p.causal && j0 + BKV - 1 > q0) || (j0 + BKV > p.N);
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        const int q = q0 + qb * 16 + fr;
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float x = s[kb][qb][r] * p.scale_log2;
            if (need_mask) {
              const int kv = j0 + kb * 16 + grp * 4 + r;
              if (kv >= p.N || (p.causal && kv > q)) x = -INFINITY;
            }
            s[kb][qb][r] = x;
            mx = fmaxf(mx, x);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mn = fmaxf(m[qb], mx);
        const float ms = (mn == -INFINITY) ? 0.f : mn;
        const float alpha = fast_exp2(m[qb] - ms);
        m[qb] = mn;
        float ps = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float w = fast_exp2(s[kb][qb][r] - ms);
            s[kb][qb][r] = w;
            ps += w;
          }
        lsum[qb] = lsum[qb] * alpha + ps;
#pragma unroll
        for (int i = 0; i < DB; ++i) o[i][qb] *= alpha;
      }
      // P^T fragments: k-step ks covers rows 32 ks + {4 grp .. 4 grp + 3, 16 + 4 grp ..}.
      bf16x8_t pf[2][2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          u32x4 w;
          w[0] = pack2(s[2 * ks][qb][0], s[2 * ks][qb][1]);
          w[1] = pack2(s[2 * ks][qb][2], s[2 * ks][qb][3]);
          w[2] = pack2(s[2 * ks + 1][qb][0], s[2 * ks + 1][qb][1]);
          w[3] = pack2(s[2 * ks + 1][qb][2], s[2 * ks + 1][qb][3]);
          pf[qb][ks] = __builtin_bit_cast(bf16x8_t, w);
        }
      // O^T[d][q] += V^T P^T: A = value column d = 16 db + fr over the same rows.
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const uint16_t* col = vt + (db * 16 + fr) * L::VT_LD + ks * 32 + grp * 4;
          const u32x2 lo = *reinterpret_cast<const u32x2*>(col);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(col + 16);
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, u32x4{lo[0], lo[1], hi[0], hi[1]});
          o[db][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pf[0][ks], o[db][0], 0, 0, 0);
          o[db][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pf[1][ks], o[db][1], 0, 0, 0);
        }
      }
    }
    if (jt + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // Normalise and store: lane holds O[q][16 db + 4 grp + r] for its query rows.
  uint16_t* __restrict__ O = reinterpret_cast<uint16_t*>(p.out);
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    float l = lsum[qb];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const int q = q0 + qb * 16 + fr;
    if (q < p.N) {
      uint16_t* dst = O + ((size_t)b * p.N + q) * p.o_stride + (size_t)h * D + grp * 4;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const u32x2 w{pack2(o[db][qb][0] * inv, o[db][qb][1] * inv),
                      pack2(o[db][qb][2] * inv, o[db][qb][3] * inv)};
        *reinterpret_cast<u32x2*>(dst + db * 16) = w;
      }
    }
  }
}

template <int D>
hipError_t launch_attn(const AttnParams& p, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)attn_bf16_kernel<D>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)AttnLds<D>::BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  dim3 grid((p.N + BQ - 1) / BQ, p.H, p.B);
  hipLaunchKernelGGL(attn_bf16_kernel<D>, grid, dim3(kThreads), AttnLds<D>::BYTES, st, p);
  return hipGetLastError();
}

}  // namespace

bool attn_bf16_supported(const AttnParams& p) {
  return p.dtype == KL_BF16 && (p.D == 64 || p.D == 128) && p.q_stride % 8 == 0 &&
         p.v_stride % 8 == 0 && p.o_stride % 8 == 0;
}

hipError_t launch_prefill_attention(const AttnParams& p, hipStream_t st) {
  if (p.N == 0 || p.B == 0) return hipSuccess;
  if (p.D == 128) return launch_attn<128>(p, st);
  if (p.D == 64) return launch_attn<64>(p, st);
  return hipErrorInvalidValue;
}

}  // namespace kl
