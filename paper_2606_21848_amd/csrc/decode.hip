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
// With one split per sequence (enough (b, g) pairs to fill the chip) a wide
// workgroup of 8 waves walks the whole cache of its pair and writes the output
// directly. Otherwise each split emits (acc[D], m, l) in fp32 to the workspace
// and decode_combine merges the splits of each (b, h) in split order.

#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

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

template <typename T>
__device__ __forceinline__ void store_out(void* out, size_t i, float v) {
  if constexpr (sizeof(T) == 2)
    reinterpret_cast<uint16_t*>(out)[i] = (uint16_t)f32_to_bf16(v);
  else
    reinterpret_cast<float*>(out)[i] = v;
}

__device__ __forceinline__ u32x4 load16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

template <typename T, int D, int R, bool PAGED, bool KEYS, int NW>
__global__ __launch_bounds__(NW * 64) void decode_partial_kernel(DecodeParams p) {
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
  const size_t bh0 = (size_t)b * p.H + g * R;  // first query head of this group
  if (start >= len) {  // uniform over the workgroup
    if (s == 0 && p.S == 1) {  // empty cache: zero output rows (the merge does this when S > 1)
      for (int i = threadIdx.x; i < R * D; i += NW * 64) store_out<T>(p.out, bh0 * D + i, 0.f);
    }
    return;
  }
  const int end = min(start + p.chunk, len);

  const int rslot = lane / LPR;        // which row of a load this lane reads
  const int col = (lane % LPR) * E;    // first element of this lane's slice

  const T* __restrict__ qp = reinterpret_cast<const T*>(p.q);
  u32x4 qv[R];
#pragma unroll
  for (int r = 0; r < R; ++r)
    qv[r] = *reinterpret_cast<const u32x4*>(qp + ((bh0 + r) * D + col));

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

  // Tile loader: this lane's U rows of the 16-row tile starting at row t0. Rows
  // past `end` (or in a block outside the cache) are clamped for the load and
  // flagged invalid; `full` says every row is valid.
  auto load_tile = [&](int t0, u32x4* v, u32x4* k, bool* valid, bool& full) {
    bool blk_ok = true;
    size_t tile_base;
    if constexpr (PAGED) {
      // The tile lies inside one block: t0 is a multiple of 16 and so is the block size.
      const int blk = p.table[(size_t)b * p.max_blocks + (t0 >> p.block_shift)];
      blk_ok = (blk >= 0) && (blk < p.num_blocks);
      tile_base = ((size_t)(blk_ok ? blk : 0) * p.G + g) << p.block_shift;
    } else {
      tile_base = (size_t)(b * p.G + g) * p.L_max;
    }
    full = blk_ok && (t0 + kTile <= end);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      int tok = t0 + u * RPL + rslot;
      valid[u] = blk_ok && (tok < end);
      if (!full) tok = min(tok, end - 1);
      const int in_blk = PAGED ? (tok & bs_mask) : tok;
      const size_t off = (tile_base + in_blk) * D + col;
      v[u] = load16(vbase + off);
      if constexpr (KEYS) k[u] = load16(kbase + off);
    }
  };

  // Two tiles in flight per wave: the next tile's loads are issued before the
  // current tile is consumed.
  u32x4 v[U], k[U], vn[U], kn[U];
  bool valid[U], validn[U];
  bool full = true, fulln = true;
  int t0 = start + wave * kTile;
  if (t0 < end) load_tile(t0, v, k, valid, full);
  for (; t0 < end; t0 += NW * kTile) {
    const int t1 = t0 + NW * kTile;
    if (t1 < end) load_tile(t1, vn, kn, validn, fulln);
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
#pragma unroll
    for (int u = 0; u < U; ++u) {
      v[u] = vn[u];
      if constexpr (KEYS) k[u] = kn[u];
      valid[u] = validn[u];
    }
    full = fulln;
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

  __shared__ float s_acc[NW][R][D];
  __shared__ float s_ml[NW][R][2];
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
  for (int i = threadIdx.x; i < R * (D + 2); i += NW * 64) {
    const int r = i / (D + 2);
    const int c = i % (D + 2);
    float mm = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) mm = fmaxf(mm, s_ml[w][r][0]);
    const float ms = (mm == -INFINITY) ? 0.f : mm;
    float lsum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) lsum += s_ml[w][r][1] * fast_exp2(s_ml[w][r][0] - ms);
    float val;
    if (c < D) {
      val = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) val += s_acc[w][r][c] * fast_exp2(s_ml[w][r][0] - ms);
    } else {
      val = (c == D) ? mm : lsum;
    }
    if (p.S == 1) {
      if (c < D) store_out<T>(p.out, (bh0 + r) * D + c, lsum > 0.f ? val / lsum : 0.f);
    } else {
      p.part[((bh0 + r) * p.S + s) * (D + 2) + c] = val;
    }
  }
}

// Merge the splits of one (b, h): weights 2^(m_s - M) / L per split, then the
// weighted sum of the split accumulators, split by split in order.
template <typename T, int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeParams p) {
  constexpr int SUB = 256 / D;  // split subsets summed in parallel per column
  __shared__ float s_w[kMaxSplits];
  __shared__ float s_red[4];
  __shared__ float s_acc[SUB][D];
  const int bh = blockIdx.x;
  const int b = bh / p.H;
  const int t = threadIdx.x;
  const int cap = p.paged ? (p.max_blocks << p.block_shift) : p.L_max;
  const int len = min(max(p.lengths[b], 0), cap);
  const int ns = (len + p.chunk - 1) / p.chunk;
  const float* __restrict__ part = p.part + (size_t)bh * p.S * (D + 2);
  if (ns == 0) {
    if (t < D) store_out<T>(p.out, (size_t)bh * D + t, 0.f);
    return;
  }
  float mloc = -INFINITY;
  for (int k = t; k < ns; k += 256) mloc = fmaxf(mloc, part[k * (D + 2) + D]);
  for (int sh = 32; sh > 0; sh >>= 1) mloc = fmaxf(mloc, __shfl_xor(mloc, sh));
  if ((t & 63) == 0) s_red[t >> 6] = mloc;
  __syncthreads();
  const float M = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
  const float Ms = (M == -INFINITY) ? 0.f : M;
  __syncthreads();
  float lloc = 0.f;
  for (int k = t; k < ns; k += 256) {
    const float w = fast_exp2(part[k * (D + 2) + D] - Ms);
    s_w[k] = w;
    lloc = fmaf(part[k * (D + 2) + D + 1], w, lloc);
  }
  for (int sh = 32; sh > 0; sh >>= 1) lloc += __shfl_xor(lloc, sh);
  if ((t & 63) == 0) s_red[t >> 6] = lloc;
  __syncthreads();
  const float L = s_red[0] + s_red[1] + s_red[2] + s_red[3];
  const int c = t % D, sub = t / D;
  float a = 0.f;
#pragma unroll 4
  for (int k = sub; k < ns; k += SUB) a = fmaf(part[k * (D + 2) + c], s_w[k], a);
  s_acc[sub][c] = a;
  __syncthreads();
  if (t < D) {
    float o = 0.f;
#pragma unroll
    for (int j = 0; j < SUB; ++j) o += s_acc[j][t];
    store_out<T>(p.out, (size_t)bh * D + t, L > 0.f ? o / L : 0.f);
  }
}

template <typename T, int D, int R, bool PAGED, bool KEYS, int NW>
hipError_t launch_t(const DecodeParams& p, hipStream_t st) {
  dim3 grid(p.S, p.G, p.B);
  if (p.ev_start) {
    hipError_t e = hipEventRecord(p.ev_start, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((decode_partial_kernel<T, D, R, PAGED, KEYS, NW>), grid, dim3(NW * 64), 0,
                     st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.ev_stop) {
    e = hipEventRecord(p.ev_stop, st);
    if (e != hipSuccess) return e;
  }
  if (p.S > 1) {
    hipLaunchKernelGGL((decode_combine_kernel<T, D>), dim3(p.B * p.H), dim3(256), 0, st, p);
    e = hipGetLastError();
  }
  return e;
}

template <typename T, int D, int R, bool PAGED, bool KEYS>
hipError_t pick_waves(const DecodeParams& p, hipStream_t st) {
  switch (p.waves) {
    case 4: return launch_t<T, D, R, PAGED, KEYS, 4>(p, st);
    case 8: return launch_t<T, D, R, PAGED, KEYS, 8>(p, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int D, int R>
hipError_t pick_layout(const DecodeParams& p, hipStream_t st) {
  const bool keys = p.kdata != nullptr;
  if (p.paged)
    return keys ? pick_waves<T, D, R, true, true>(p, st) : pick_waves<T, D, R, true, false>(p, st);
  return keys ? pick_waves<T, D, R, false, true>(p, st) : pick_waves<T, D, R, false, false>(p, st);
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
  if (p.S > kMaxSplits) return hipErrorInvalidValue;
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
