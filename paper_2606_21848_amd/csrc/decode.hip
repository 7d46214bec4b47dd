// Value-only-cache decode (Section 3) and the standard K+V comparison decode.
//
// Split-K over the cache length. A workgroup (4 waves) owns one
// (sequence b, value group g, split s) and the R = H/G query heads of that
// group. Each wave walks 16-row tiles of the split; a lane group of LPR lanes
// holds one cache row per 16-byte load, so one wave-wide load moves RPL whole
// rows (1 KiB) and the 16-row tile is U loads. The tile stays in registers and
// is used twice: for the scores s = <q~, v> (Eq. 4, dot products reduced over
// the lane group with DPP) and for the weighted sum acc += exp(s - m) v of the
// online softmax. Nothing is re-read, so a value row crosses HBM once.
//
// Each split emits (acc[D], m, l) in fp32; decode_combine merges the splits of
// one (b, h) in split order.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

constexpr int kWaves = 4;
constexpr int kTile = 16;  // rows per wave iteration

template <typename T>
struct Elem;
template <>
struct Elem<uint16_t> {
  static constexpr int E = 8;  // elements per 16-byte load
};
template <>
struct Elem<float> {
  static constexpr int E = 4;
};

// Score contribution of one 16-byte slice: dot(q, x) over E elements.
__device__ __forceinline__ float slice_dot(const u32x4& q, const u32x4& x, uint16_t) {
  float p = dot2_bf16(q.x, x.x, 0.f);
  p = dot2_bf16(q.y, x.y, p);
  p = dot2_bf16(q.z, x.z, p);
  return dot2_bf16(q.w, x.w, p);
}
__device__ __forceinline__ float slice_dot(const u32x4& q, const u32x4& x, float) {
  float p = __uint_as_float(q.x) * __uint_as_float(x.x);
  p = fmaf(__uint_as_float(q.y), __uint_as_float(x.y), p);
  p = fmaf(__uint_as_float(q.z), __uint_as_float(x.z), p);
  return fmaf(__uint_as_float(q.w), __uint_as_float(x.w), p);
}

__device__ __forceinline__ void slice_to_f32(const u32x4& x, float* f, uint16_t) {
  f[0] = bf16_lo(x.x); f[1] = bf16_hi(x.x);
  f[2] = bf16_lo(x.y); f[3] = bf16_hi(x.y);
  f[4] = bf16_lo(x.z); f[5] = bf16_hi(x.z);
  f[6] = bf16_lo(x.w); f[7] = bf16_hi(x.w);
}
__device__ __forceinline__ void slice_to_f32(const u32x4& x, float* f, float) {
  f[0] = __uint_as_float(x.x); f[1] = __uint_as_float(x.y);
  f[2] = __uint_as_float(x.z); f[3] = __uint_as_float(x.w);
}

__device__ __forceinline__ u32x4 load16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

template <typename T, int D, int R, bool PAGED, bool KEYS>
__global__ __launch_bounds__(kWaves * 64) void decode_partial_kernel(DecodeParams p) {
  constexpr int E = Elem<T>::E;
  constexpr int LPR = D / E;     // lanes per cache row
  constexpr int RPL = 64 / LPR;  // rows per wave-wide load
  constexpr int U = kTile / RPL; // loads per tile
  static_assert(RPL * U == kTile, "tile shape");

  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cap = PAGED ? (p.max_blocks << p.block_shift) : p.L_max;
  const int len = min(max(p.lengths[b], 0), cap);
  const int start = s * p.chunk;
  if (start >= len) return;  // uniform over the workgroup
  const int end = min(start + p.chunk, len);

  const int rslot = lane / LPR;        // which row of a load this lane reads
  const int col = (lane % LPR) * E;    // first element of this lane's slice

  const T* __restrict__ qp = reinterpret_cast<const T*>(p.q);
  u32x4 qv[R];
#pragma unroll
  for (int r = 0; r < R; ++r)
    qv[r] = *reinterpret_cast<const u32x4*>(qp + ((size_t)(b * p.H + g * R + r) * D + col));

  float m[R], l[R], acc[R][E];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[r][e] = 0.f;
  }

  const T* __restrict__ vbase = reinterpret_cast<const T*>(p.vdata);
  const T* __restrict__ kbase = reinterpret_cast<const T*>(p.kdata);
  const int bs_mask = (1 << p.block_shift) - 1;

  for (int t0 = start + wave * kTile; t0 < end; t0 += kWaves * kTile) {
    // Row offsets (in elements) of this lane's U rows.
    size_t off[U];
    bool valid[U];
    bool blk_ok = true;
    size_t tile_base = 0;
    if constexpr (PAGED) {
      // The tile lies inside one block: t0 is a multiple of 16 and so is the block size.
      const int blk = p.table[(size_t)b * p.max_blocks + (t0 >> p.block_shift)];
      blk_ok = (blk >= 0) && (blk < p.num_blocks);
      tile_base = ((size_t)(blk_ok ? blk : 0) * p.G + g) << p.block_shift;
    } else {
      tile_base = (size_t)(b * p.G + g) * p.L_max;
    }
    const bool full = blk_ok && (t0 + kTile <= end);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      int tok = t0 + u * RPL + rslot;
      valid[u] = blk_ok && (tok < end);
      if (!full) tok = min(tok, end - 1);
      const int in_blk = PAGED ? (tok & bs_mask) : tok;
      off[u] = (tile_base + in_blk) * D + col;
    }
    u32x4 v[U];
    u32x4 k[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      v[u] = load16(vbase + off[u]);
      if constexpr (KEYS) k[u] = load16(kbase + off[u]);
    }
    if (!full) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (!valid[u]) v[u] = u32x4{0u, 0u, 0u, 0u};  // padding may hold NaN
    }
    float vf[U][E];
#pragma unroll
    for (int u = 0; u < U; ++u) slice_to_f32(v[u], vf[u], T());

#pragma unroll
    for (int r = 0; r < R; ++r) {
      float sc[U];
      float mt = m[r];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float part = slice_dot(qv[r], KEYS ? k[u] : v[u], T());
        float x = group_sum<LPR>(part) * p.scale_log2;
        if (!full && !valid[u]) x = -INFINITY;
        sc[u] = x;
        mt = fmaxf(mt, x);
      }
      const float ms = (mt == -INFINITY) ? 0.f : mt;
      const float alpha = fast_exp2(m[r] - ms);
      float lsum = l[r] * alpha;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[r][e] *= alpha;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float w = fast_exp2(sc[u] - ms);
        lsum += w;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[r][e] = fmaf(w, vf[u][e], acc[r][e]);
      }
      l[r] = lsum;
      m[r] = mt;
    }
  }

  // Merge the RPL row slots of the wave (lanes LPR apart), then the waves.
#pragma unroll
  for (int sh = LPR; sh < 64; sh <<= 1) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float m2 = __shfl_xor(m[r], sh);
      const float l2 = __shfl_xor(l[r], sh);
      float f1, f2, mm;
      merge_scale(m[r], m2, f1, f2, mm);
      l[r] = l[r] * f1 + l2 * f2;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float a2 = __shfl_xor(acc[r][e], sh);
        acc[r][e] = acc[r][e] * f1 + a2 * f2;
      }
      m[r] = mm;
    }
  }

  __shared__ float s_acc[kWaves][R][D];
  __shared__ float s_ml[kWaves][R][2];
  if (lane < LPR) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
      for (int e = 0; e < E; ++e) s_acc[wave][r][col + e] = acc[r][e];
      if (lane == 0) {
        s_ml[wave][r][0] = m[r];
        s_ml[wave][r][1] = l[r];
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < R * (D + 2); i += kWaves * 64) {
    const int r = i / (D + 2);
    const int c = i % (D + 2);
    float mm = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mm = fmaxf(mm, s_ml[w][r][0]);
    const float ms = (mm == -INFINITY) ? 0.f : mm;
    float val = 0.f;
    if (c < D) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) val += s_acc[w][r][c] * fast_exp2(s_ml[w][r][0] - ms);
    } else if (c == D) {
      val = mm;
    } else {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) val += s_ml[w][r][1] * fast_exp2(s_ml[w][r][0] - ms);
    }
    const size_t bh = (size_t)b * p.H + g * R + r;
    p.part[(bh * p.S + s) * (D + 2) + c] = val;
  }
}

template <typename T, int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(DecodeParams p) {
  const int bh = blockIdx.x;
  const int b = bh / p.H;
  const int c = threadIdx.x;
  const int cap = p.paged ? (p.max_blocks << p.block_shift) : p.L_max;
  const int len = min(max(p.lengths[b], 0), cap);
  const int ns = (len + p.chunk - 1) / p.chunk;
  const float* __restrict__ part = p.part + (size_t)bh * p.S * (D + 2);
  float mm = -INFINITY;
  for (int s = 0; s < ns; ++s) mm = fmaxf(mm, part[s * (D + 2) + D]);
  float o = 0.f;
  if (mm != -INFINITY) {
    float lsum = 0.f, a = 0.f;
    for (int s = 0; s < ns; ++s) {
      const float f = fast_exp2(part[s * (D + 2) + D] - mm);
      lsum = fmaf(part[s * (D + 2) + D + 1], f, lsum);
      a = fmaf(part[s * (D + 2) + c], f, a);
    }
    o = a / lsum;
  }
  if constexpr (sizeof(T) == 2) {
    reinterpret_cast<uint16_t*>(p.out)[(size_t)bh * D + c] = (uint16_t)f32_to_bf16(o);
  } else {
    reinterpret_cast<float*>(p.out)[(size_t)bh * D + c] = o;
  }
}

template <typename T, int D, int R, bool PAGED, bool KEYS>
hipError_t launch_t(const DecodeParams& p, hipStream_t st) {
  dim3 grid(p.S, p.G, p.B);
  if (p.ev_start) {
    hipError_t e = hipEventRecord(p.ev_start, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((decode_partial_kernel<T, D, R, PAGED, KEYS>), grid, dim3(kWaves * 64), 0,
                     st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.ev_stop) {
    e = hipEventRecord(p.ev_stop, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((decode_combine_kernel<T, D>), dim3(p.B * p.H), dim3(D), 0, st, p);
  return hipGetLastError();
}

template <typename T, int D, int R>
hipError_t pick_layout(const DecodeParams& p, hipStream_t st) {
  const bool keys = p.kdata != nullptr;
  if (p.paged)
    return keys ? launch_t<T, D, R, true, true>(p, st) : launch_t<T, D, R, true, false>(p, st);
  return keys ? launch_t<T, D, R, false, true>(p, st) : launch_t<T, D, R, false, false>(p, st);
}

template <typename T, int D>
hipError_t pick_r(const DecodeParams& p, hipStream_t st) {
  switch (p.R) {
    case 1: return pick_layout<T, D, 1>(p, st);
    case 2: return pick_layout<T, D, 2>(p, st);
    case 4: return pick_layout<T, D, 4>(p, st);
    case 8: return pick_layout<T, D, 8>(p, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, hipStream_t st) {
  if (p.dtype == KL_BF16) {
    if (p.D == 128) return pick_r<uint16_t, 128>(p, st);
    if (p.D == 64) return pick_r<uint16_t, 64>(p, st);
  } else {
    if (p.D == 128) return pick_r<float, 128>(p, st);
    if (p.D == 64) return pick_r<float, 64>(p, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace kl
