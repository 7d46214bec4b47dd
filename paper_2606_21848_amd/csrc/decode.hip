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
// With one split per sequence (enough (b, g) pairs to fill the chip) the
// workgroup walks the whole cache of its pair and writes the output directly
// (four waves: eight ran 3% slower on the batch-8 step). Otherwise each split
// emits (acc[D], m, l) in fp32 to the workspace and decode_combine merges the
// splits of each (b, h) in split order.

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

__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi) {
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 b2;
  b2 x = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, x);
}

template <typename T>
__device__ __forceinline__ void store_out(void* out, size_t i, float v) {
  if constexpr (sizeof(T) == 2)
    reinterpret_cast<uint16_t*>(out)[i] = (uint16_t)f32_to_bf16(v);
  else
    reinterpret_cast<float*>(out)[i] = v;
}

typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// Stages of the per-wave LDS ring: as many as fit in 64 KiB per 4-wave
// workgroup (two per CU) or 96 KiB per 8-wave one, at least 2 and at most 4.
constexpr int stage_count(int stage_bytes, int waves) {
  const int n = (waves >= 8 ? 98304 : 65536) / (stage_bytes * waves);
  return n < 2 ? 2 : (n > 4 ? 4 : n);
}

// Shape of the per-wave staging ring: NBUF stages of one 16-row tile (V, then
// K when present), each moved by NI direct-to-LDS copy instructions of 1 KiB.
template <typename T, int D, bool KEYS, int NW>
struct Ring {
  static constexpr int ROWB = D * (int)sizeof(T);  // bytes per cache row
  static constexpr int TB = kTile * ROWB;          // bytes per tile
  static constexpr int NI = TB / 1024;             // copy instructions per tile
  static constexpr int KV = KEYS ? 2 : 1;
  static constexpr int SB = TB * KV;               // bytes per stage
  static constexpr int NBUF = stage_count(SB, NW);
  static constexpr int PER_TILE = NI * KV;         // copies per tile
  static constexpr int BYTES = NBUF * SB * NW;     // whole workgroup
};

// Streams the tiles of rows [t_first + j * step, +16) for j = 0, 1, ... below
// `end` through this wave's LDS ring and hands each landed tile to
// consume(stage, t0, blk_ok). Copy instruction i of a tile moves its bytes
// [1024 i, 1024 i + 1024): lane L lands at byte 1024 i + 16 L, i.e. row rr,
// slot sl, and fetches logical chunk sl ^ swz(rr) of that row, so the consumer
// finds chunk c of row rr at slot c ^ swz(rr). Rows past `end` are clamped to
// the last row; a block id outside the cache reads block 0 and is reported as
// blk_ok = false. `ready` runs once after the first copies are issued.
template <typename T, int D, bool PAGED, bool KEYS, int NW, class Swz, class Ready, class Consume>
__device__ __forceinline__ void stream_tiles(const DecodeParams& p, int b, int g, int lane,
                                             lds_u8* ring, int t_first, int end, Swz swz,
                                             Ready ready, Consume consume) {
  using RS = Ring<T, D, KEYS, NW>;
  constexpr int ROWB = RS::ROWB, TB = RS::TB, NI = RS::NI, SB = RS::SB, NBUF = RS::NBUF;
  constexpr int PER_TILE = RS::PER_TILE;
  const int step = NW * kTile;
  const int ntiles = (t_first < end) ? (end - t_first + step - 1) / step : 0;  // uniform
  if (ntiles == 0) return;
  const uint32_t ring_addr = (uint32_t)(uintptr_t)ring;

  int cp_row[NI];       // tile row this lane copies, per instruction
  uint32_t cp_col[NI];  // byte offset of the fetched chunk within the row
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int pos = i * 1024 + 16 * lane;
    cp_row[i] = pos / ROWB;
    cp_col[i] = (uint32_t)((((pos % ROWB) / 16) ^ swz(pos / ROWB)) * 16);
  }
  const unsigned char* __restrict__ vbytes = reinterpret_cast<const unsigned char*>(p.vdata);
  const unsigned char* __restrict__ kbytes = reinterpret_cast<const unsigned char*>(p.kdata);
  const int bs_mask = (1 << p.block_shift) - 1;
  // The table is read through the constant address space so the uniform
  // lookups stay scalar loads (the copies' memory clobbers would otherwise turn
  // them into vector loads whose waits drain the copy pipeline).
  const __attribute__((address_space(4))) int* table =
      (const __attribute__((address_space(4))) int*)p.table;
  auto block_of = [&](int t) -> int {
    if constexpr (PAGED) return table[(size_t)b * p.max_blocks + (t >> p.block_shift)];
    return 0;
  };
  auto block_ok = [&](int blk) { return !PAGED || (blk >= 0 && blk < p.num_blocks); };
  auto issue = [&](int j, int blk) {
    const int t = t_first + j * step;
    size_t row0;
    if constexpr (PAGED)  // the tile lies inside one block (both are multiples of 16 rows)
      row0 = (((size_t)(block_ok(blk) ? blk : 0) * p.G + g) << p.block_shift) + (t & bs_mask);
    else
      row0 = (size_t)(b * p.G + g) * p.L_max + t;
    const int last = end - 1 - t;
    const uint32_t st = ring_addr + (uint32_t)((j % NBUF) * SB);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const uint32_t off = (uint32_t)(min(cp_row[i], last) * ROWB) + cp_col[i];
      copy_to_lds_nt(vbytes + row0 * ROWB, off, st + i * 1024);
      if constexpr (KEYS) copy_to_lds_nt(kbytes + row0 * ROWB, off, st + TB + i * 1024);
    }
  };

  int bq[NBUF];  // block ids of tiles j .. j + NBUF - 1 (constant indices: scalar registers)
#pragma unroll
  for (int i = 0; i < NBUF; ++i) bq[i] = 0;
#pragma unroll
  for (int i = 0; i < NBUF - 1; ++i) {
    if (i < ntiles) {
      bq[i] = block_of(t_first + i * step);
      issue(i, bq[i]);
    }
  }
  ready();
  // Tiles j+1 .. j+NBUF-1 stay in flight while tile j is consumed. The wait
  // before tile j allows only the copies issued after it to be outstanding;
  // the vector memory counter retires in issue order, so tile j has landed.
  for (int j = 0; j < ntiles; ++j) {
    const int jn = j + NBUF - 1;
    const int ahead = min(NBUF - 1, ntiles - 1 - j);  // tiles issued after tile j
    if (jn < ntiles) {
      // The stage being refilled was consumed in the previous iteration: its
      // LDS reads have completed before the copies may overwrite it.
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      bq[NBUF - 1] = block_of(t_first + jn * step);
      issue(jn, bq[NBUF - 1]);
    }
    switch (ahead) {
      case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
      case 1: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(PER_TILE) : "memory"); break;
      case 2: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * PER_TILE) : "memory"); break;
      default: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * PER_TILE) : "memory"); break;
    }
    consume(ring + (j % NBUF) * SB, t_first + j * step, block_ok(bq[0]));
#pragma unroll
    for (int i = 0; i < NBUF - 1; ++i) bq[i] = bq[i + 1];
  }
}

// Where a finished segment goes: the normalised output rows of its heads
// (part == nullptr), or one partial row (acc[D], m, l) per head, `stride`
// floats apart.
struct SegOut {
  float* part;
  int stride;
};

// Merge the per-wave states (acc[R][D] of wave w at s_acc + w WS, m and l in
// s_ml) of the workgroup and store them to `o`. Ends with a barrier, so the LDS
// can be refilled.
template <typename T, int D, int R, int NW, int WS = R * D>
__device__ __forceinline__ void merge_waves(const DecodeParams& p, const float* s_acc,
                                            const float (*s_ml)[R][2], size_t bh0, SegOut o) {
  // Per head, once: the common reference (the largest wave maximum), each
  // wave's factor 2^(m_w - reference) and the merged weight sum.
  __shared__ float s_f[NW][R];
  __shared__ float s_h[R][2];
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += NW * 64) {
    float mm = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) mm = fmaxf(mm, s_ml[w][r][0]);
    const float ms = (mm == -INFINITY) ? 0.f : mm;
    float lsum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = fast_exp2(s_ml[w][r][0] - ms);  // 0 for a wave that saw no row
      s_f[w][r] = f;
      lsum += s_ml[w][r][1] * f;
    }
    s_h[r][0] = mm;
    s_h[r][1] = lsum;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < R * (D + 2); i += NW * 64) {
    const int r = i / (D + 2);
    const int c = i % (D + 2);
    const float lsum = s_h[r][1];
    float val;
    if (c < D) {
      val = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) val += s_acc[w * WS + r * D + c] * s_f[w][r];
    } else {
      val = (c == D) ? s_h[r][0] : lsum;
    }
    if (o.part == nullptr) {
      if (c < D) store_out<T>(p.out, (bh0 + r) * D + c, lsum > 0.f ? val / lsum : 0.f);
    } else {
      o.part[(size_t)r * o.stride + c] = val;
    }
  }
  __syncthreads();
}

// Rows decoded for sequence b (the new row included when the step appends),
// clamped to the cache capacity.
// The lengths (and the plan) are read through the constant address space:
// nothing in the kernel writes them, and the uniform reads then stay scalar
// loads even where the kernel stores to other global memory (the appended row).
__device__ __forceinline__ int length_of(const DecodeParams& p, int b) {
  return ((const __attribute__((address_space(4))) int*)p.lengths)[b];
}
__device__ __forceinline__ int decode_rows(const DecodeParams& p, int b, int cap) {
  return min(max(length_of(p, b) + (p.vnew ? 1 : 0), 0), cap);
}
template <bool PAGED>
__device__ __forceinline__ int seq_len(const DecodeParams& p, int b) {
  return decode_rows(p, b, PAGED ? (p.max_blocks << p.block_shift) : p.L_max);
}

// The step's new row of pair (b, g), when this segment [start, end) holds it:
// its position, else -1. The new row is the last decoded row of the sequence;
// past the capacity it is dropped (and not decoded), as an append drops it.
template <bool PAGED>
__device__ __forceinline__ int new_row_in(const DecodeParams& p, int b, int start, int end) {
  if (!p.vnew) return -1;
  const int cap = PAGED ? (p.max_blocks << p.block_shift) : p.L_max;
  const int pos = length_of(p, b);
  return (pos >= 0 && pos < cap && pos >= start && pos < end) ? pos : -1;
}

// The step's new value row of pair (b, g): lane i < ROWB / 16 holds its 16-byte
// chunk i. Loaded before the cached rows stream, so its latency is hidden.
template <typename T, int D>
__device__ __forceinline__ u32x4 load_new_row(const DecodeParams& p, int b, int g, int lane) {
  constexpr int CH = D * (int)sizeof(T) / 16;
  const u32x4* src = reinterpret_cast<const u32x4*>(
      reinterpret_cast<const unsigned char*>(p.vnew) + ((size_t)b * p.G + g) * CH * 16);
  return lane < CH ? src[lane] : u32x4{0u, 0u, 0u, 0u};
}

// Appends the new row (held as by load_new_row) to the cache at row pos, and
// stages it as row 0 of a tile in LDS with the other rows zero, so that masked
// rows contribute exact zeros to any product. One wave; the stage must be idle.
template <typename T, int D, bool PAGED>
__device__ __forceinline__ void append_and_stage(const DecodeParams& p, int b, int g, int pos,
                                                 u32x4 chunk, lds_u8* stage, int lane) {
  constexpr int CH = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  for (int i = lane; i < kTile * CH; i += 64)
    *reinterpret_cast<__attribute__((address_space(3))) u32x4*>(stage + i * 16) =
        i < CH ? chunk : u32x4{0u, 0u, 0u, 0u};
  size_t row;
  bool ok = true;
  if constexpr (PAGED) {
    const int blk = p.table[(size_t)b * p.max_blocks + (pos >> p.block_shift)];
    ok = blk >= 0 && blk < p.num_blocks;
    row = ((((size_t)(ok ? blk : 0)) * p.G + g) << p.block_shift) + (pos & ((1 << p.block_shift) - 1));
  } else {
    row = ((size_t)b * p.G + g) * p.L_max + pos;
  }
  if (ok && lane < CH)
    reinterpret_cast<u32x4*>(p.vdata)[row * CH + lane] = chunk;
}

// Runs seg(b, g, row_begin, row_end, out) for every segment this workgroup owns.
//
// Split mode: the grid is (S, G, B) and workgroup (s, g, b) owns rows
// [s chunk, (s+1) chunk) of pair (b, g); with one split it stores the output
// rows, otherwise partial s of each head.
//
// Balanced mode: the 16-row tiles of all pairs, pair (b, g) after (b, g-1) and
// sequence b after b-1, form one sequence of T tiles, and workgroup w owns
// tiles [w per, (w+1) per) with per = ceil(T / workgroups), which may cross
// pairs. A pair that lies inside one workgroup stores its output rows;
// otherwise each workgroup on it stores a partial at index pair + w, which is
// unique (along the tile sequence both the pair and the workgroup index are
// non-decreasing and at least one grows from one segment to the next).
// Balanced mode over at most kWavePlanMax sequences runs no plan kernel: a
// wave derives the plan from the lengths, one sequence per lane. n = the
// lane's tiles (zero past B), pre = the exclusive prefix sum of n over the
// sequences before it, sum = the tiles of all sequences (uniform).
constexpr int kWavePlanMax = 64;
struct LanePlan {
  int n, pre, sum;
};
__device__ __forceinline__ LanePlan lane_plan(const DecodeParams& p, int cap) {
  const int lane = threadIdx.x & 63;
  const int n = lane < p.B ? (decode_rows(p, lane, cap) + kTile - 1) / kTile : 0;
  int incl = n;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(incl, off, 64);
    if (lane >= off) incl += v;
  }
  return {n, incl - n, __builtin_amdgcn_readlane(incl, 63)};
}

template <typename T, int D, int R, bool PAGED, int NW, class Seg>
__device__ __forceinline__ void for_each_segment(const DecodeParams& p, Seg seg) {
  if (!p.balanced) {
    const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int len = seq_len<PAGED>(p, b);
    const int start = s * p.chunk;
    const size_t bh0 = (size_t)b * p.H + g * R;
    if (start >= len) {  // uniform over the workgroup
      if (s == 0 && p.S == 1) {  // empty cache: zero output rows (the merge does this when S > 1)
        for (int i = threadIdx.x; i < R * D; i += NW * 64) store_out<T>(p.out, bh0 * D + i, 0.f);
      }
      return;
    }
    const SegOut o = p.S == 1 ? SegOut{nullptr, 0}
                              : SegOut{p.part + (bh0 * p.S + s) * (D + 2), p.S * (D + 2)};
    seg(b, g, start, min(start + p.chunk, len), o);
    return;
  }
  const __attribute__((address_space(4))) int* plan = (const __attribute__((address_space(4))) int*)p.plan;
  const __attribute__((address_space(4))) int* pre = plan + 2;  // exclusive prefix sums of tiles, [B + 1]
  const bool wave_planned = p.B <= kWavePlanMax;  // uniform
  const int cap = PAGED ? (p.max_blocks << p.block_shift) : p.L_max;
  int total, per;
  LanePlan lp{};
  if (wave_planned) {
    lp = lane_plan(p, cap);
    total = p.G * lp.sum;
    per = total > 0 ? (total + p.nwg - 1) / p.nwg : 1;
  } else {
    total = plan[0];
    per = plan[1];
  }
  const int w = blockIdx.x;
  int t = w * per;
  const int t_end = min(total, t + per);
  if (t >= t_end) return;
  // Sequence holding tile t: the last b with G * pre[b] <= t (empty sequences
  // share their start with the next one and are skipped by taking the last),
  // and pre[b], carried along as the walk moves to later sequences.
  int b, preb;
  if (wave_planned) {
    const unsigned long long below = __ballot((int)(threadIdx.x & 63) < p.B && p.G * lp.pre <= t);
    b = 63 - __clzll((long long)below);  // tile 0 lies in sequence 0 or later: below != 0
    preb = __builtin_amdgcn_readlane(lp.pre, b);
  } else {
    int lo = 0, hi = p.B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (p.G * pre[mid] <= t) lo = mid; else hi = mid - 1;
    }
    b = lo;
    preb = pre[b];
  }
  auto tiles_of = [&](int bb) {  // tiles per pair of sequence bb
    return wave_planned ? (seq_len<PAGED>(p, bb) + kTile - 1) / kTile : pre[bb + 1] - pre[bb];
  };
  while (t < t_end) {
    const int n = tiles_of(b);  // > 0 here
    const int base = p.G * preb;
    const int g = (t - base) / n;
    const int tp = base + g * n;  // first tile of pair (b, g)
    const int seg_end = min(t_end, tp + n);
    const int len = seq_len<PAGED>(p, b);
    const bool whole = (tp / per) == ((tp + n - 1) / per);
    const int pair = b * p.G + g;
    const SegOut o = whole ? SegOut{nullptr, 0}
                           : SegOut{p.part + (size_t)(pair + w) * R * (D + 2), D + 2};
    seg(b, g, (t - tp) * kTile, min((seg_end - tp) * kTile, len), o);
    t = seg_end;
    if (t >= base + p.G * n) {  // past the last pair of b: next non-empty sequence
      preb += n;
      ++b;
      while (b < p.B && tiles_of(b) == 0) ++b;
    }
  }
}

// Vector-ALU consumer. A lane group of LPR lanes holds one cache row per
// 16-byte chunk, so one wave-wide LDS read covers RPL rows and a tile is U
// reads. The tile is used twice: for the scores s = <q~, v> (dot products
// reduced over the lane group with DPP) and for acc += 2^(s - m) v.
template <typename T, int D, int R, bool PAGED, bool KEYS, int NW>
__global__ __launch_bounds__(NW * 64) void decode_partial_kernel(DecodeParams p) {
  constexpr int EC = Elem<T>::E;  // elements per 16-byte chunk
  constexpr int NC = D / EC;      // chunks per cache row
  constexpr int LPR = NC;         // lanes per cache row
  constexpr int RPL = 64 / LPR;   // rows per wave-wide read
  constexpr int U = kTile / RPL;  // rows per lane per tile
  constexpr int E = EC;           // elements per lane per row
  static_assert(RPL * U == kTile, "tile shape");
  using RS = Ring<T, D, KEYS, NW>;
  constexpr int ROWB = RS::ROWB, TB = RS::TB, NBUF = RS::NBUF, SB = RS::SB;
  // Grouped heads over a bf16 cache take the lazy-reference / bf16-dot path.
  constexpr bool kGroupedBf16 = (R >= 2) && (sizeof(T) == 2) && (U % 2 == 0);
  constexpr float kLazy = 8.f;  // log2 headroom before the reference moves

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rslot = lane / LPR;  // which row of a read this lane takes
  const int lc = lane % LPR;     // this lane's chunk
  extern __shared__ __attribute__((aligned(1024))) unsigned char dyn_lds[];
  lds_u8* const ring = (lds_u8*)dyn_lds + wave * (NBUF * SB);
  __shared__ float s_acc[NW][R][D];
  __shared__ float s_ml[NW][R][2];

  auto segment = [&](int b, int g, int start, int end, SegOut so) {
  const size_t bh0 = (size_t)b * p.H + g * R;
  const T* __restrict__ qp = reinterpret_cast<const T*>(p.q);
  u32x4 qv[R];
#pragma unroll
  for (int r = 0; r < R; ++r) qv[r] = *reinterpret_cast<const u32x4*>(qp + ((bh0 + r) * D + lc * EC));

  float m[R], l[R], acc[R][E];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[r][e] = 0.f;
  }

  auto swz = [](int) { return 0; };  // one row per 16-lane pass: no conflicts
  // Take the query loads' wait once, outside the tile loop.
  auto ready = [&]() {
#pragma unroll
    for (int r = 0; r < R; ++r) asm volatile("" ::"v"(qv[r]));
  };

  // Rows at or past vend are masked: the segment's end, or the new row's
  // position while the cached rows stream when the step appends.
  int vend = end;
  auto consume = [&](const lds_u8* stage, int t0, bool blk_ok) {
    const bool full = blk_ok && (t0 + kTile <= vend);
    u32x4 v[U], k[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int rr = u * RPL + rslot;
      valid[u] = blk_ok && (t0 + rr < vend);
      const int off = rr * ROWB + lc * 16;
      v[u] = *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(stage + off);
      if constexpr (KEYS)
        k[u] = *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(stage + TB + off);
    }
    if (!full) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (!valid[u]) v[u] = u32x4{0u, 0u, 0u, 0u};  // clamped rows, or a block outside the cache
    }
    // Scores: dot products over the lane's elements, summed over the LPR lanes
    // of the row (DPP), scaled to log2 units; invalid rows get -inf.
    float sc[R][U];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float x = group_sum<LPR>(slice_dot(qv[r], KEYS ? k[u] : v[u], T())) * p.scale_log2;
        if (!full && !valid[u]) x = -INFINITY;
        sc[r][u] = x;
      }
    if constexpr (kGroupedBf16) {
      // A lazily moved reference exponent per head (raised only when a score
      // exceeds it by 2^8, so the rescale of acc is rare and weights stay below
      // 256), and the weighted sum as bf16 dot products over row pairs:
      // (w_u0, w_u1) . (v_u0[e], v_u1[e]).
      float tmax[R];
      bool grow = false;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        tmax[r] = sc[r][0];
#pragma unroll
        for (int u = 1; u < U; ++u) tmax[r] = fmaxf(tmax[r], sc[r][u]);
        grow |= tmax[r] > m[r] + kLazy;
      }
      if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const float mn = (tmax[r] > m[r] + kLazy) ? tmax[r] : m[r];
          const float alpha = (m[r] == -INFINITY) ? 0.f : fast_exp2(m[r] - mn);
          l[r] *= alpha;
#pragma unroll
          for (int e = 0; e < E; ++e) acc[r][e] *= alpha;
          m[r] = mn;
        }
      }
      uint32_t lo[U / 2][4], hi[U / 2][4];
#pragma unroll
      for (int pr = 0; pr < U / 2; ++pr)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          lo[pr][j] = __builtin_amdgcn_perm(v[2 * pr + 1][j], v[2 * pr][j], 0x05040100u);
          hi[pr][j] = __builtin_amdgcn_perm(v[2 * pr + 1][j], v[2 * pr][j], 0x07060302u);
        }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const float nm = (m[r] == -INFINITY) ? 0.f : -m[r];
        float w[U];
        float ls = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          w[u] = fast_exp2(sc[r][u] + nm);
          ls += w[u];
        }
        l[r] += ls;
#pragma unroll
        for (int pr = 0; pr < U / 2; ++pr) {
          const uint32_t wp = pack_bf16_rne(w[2 * pr], w[2 * pr + 1]);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            acc[r][2 * j] = dot2_bf16(wp, lo[pr][j], acc[r][2 * j]);
            acc[r][2 * j + 1] = dot2_bf16(wp, hi[pr][j], acc[r][2 * j + 1]);
          }
        }
      }
    } else {
      float vf[U][E];
#pragma unroll
      for (int u = 0; u < U; ++u) slice_to_f32(v[u], vf[u], T());
#pragma unroll
      for (int r = 0; r < R; ++r) {
        float mt = m[r];
#pragma unroll
        for (int u = 0; u < U; ++u) mt = fmaxf(mt, sc[r][u]);
        const float ms = (mt == -INFINITY) ? 0.f : mt;
        const float alpha = fast_exp2(m[r] - ms);
        float lsum = l[r] * alpha;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[r][e] *= alpha;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const float w = fast_exp2(sc[r][u] - ms);
          lsum += w;
#pragma unroll
          for (int e = 0; e < E; ++e) acc[r][e] = fmaf(w, vf[u][e], acc[r][e]);
        }
        l[r] = lsum;
        m[r] = mt;
      }
    }
  };

  const int pnew = KEYS ? -1 : new_row_in<PAGED>(p, b, start, end);
  if (pnew >= 0) vend = pnew;
  const u32x4 nrow = (pnew >= 0) ? load_new_row<T, D>(p, b, g, lane) : u32x4{0u, 0u, 0u, 0u};
  stream_tiles<T, D, PAGED, KEYS, NW>(p, b, g, lane, ring, start + wave * kTile, vend, swz, ready,
                                      consume);
  if (pnew >= 0 && wave == 0) {  // the step's new row: from registers, not from the cache
    append_and_stage<T, D, PAGED>(p, b, g, pnew, nrow, ring, lane);
    vend = pnew + 1;
    consume(ring, pnew, true);
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
  if (lane < LPR) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
      for (int j = 0; j < EC; ++j) s_acc[wave][r][lc * EC + j] = acc[r][j];
      if (lane == 0) {
        s_ml[wave][r][0] = m[r];
        s_ml[wave][r][1] = l[r];
      }
    }
  }
  merge_waves<T, D, R, NW>(p, &s_acc[0][0][0], s_ml, bh0, so);
  };
  for_each_segment<T, D, R, PAGED, NW>(p, segment);
}

// Matrix-core consumer for grouped heads over a 128-wide bf16 cache (R >= 2).
// Per 16-row tile, with the R heads of the group as the N = 16 columns of
// ceil(R / 16) column blocks (unused columns zero; every block reuses the same
// LDS operand reads):
//   scores   S[row][h]  = sum_d V[row][d] q~[h][d]       4 x MFMA 16x16x32,
//   weights  P[row][h]  = 2^(S - m_h)  (lazy reference m_h, as above),
//   output   O^T[d][h] += sum_row V^T[d][row] P[row][h]  8 x MFMA 16x16x16.
// The score result already has the layout of the second product's B operand
// (lane l: rows 4 (l/16) + i, head l % 16), and V^T comes from transposing LDS
// reads of the same staged tile, so every value row is still read from HBM
// once. Tile rows are XOR-swizzled by f(r) = ((r & 7) << 1) | (r >> 3) over
// the 16 chunks of a row: the score reads (16 rows, one chunk) and the
// transposing reads (8 rows, two chunks per pass) hit disjoint banks.
template <int R, bool PAGED, bool KEYS, int NW>
__global__ __launch_bounds__(NW * 64) void decode_mfma_kernel(DecodeParams p) {
  using T = uint16_t;
  constexpr int D = 128;
  using RS = Ring<T, D, KEYS, NW>;
  constexpr int TB = RS::TB, NBUF = RS::NBUF, SB = RS::SB;
  constexpr float kLazy = 8.f;
  static_assert(R >= 2 && R <= 32, "heads per group");
  constexpr int NB = (R + 15) / 16;  // 16-head column blocks

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = lane >> 4;  // lane group: rows 4 grp .. 4 grp + 3 of a score tile
  const int hl = lane & 15;   // head (column) of this lane in the score / output tiles
  auto fsw = [](int r) { return ((r & 7) << 1) | ((r >> 3) & 1); };
  extern __shared__ __attribute__((aligned(1024))) unsigned char dyn_lds[];
  lds_u8* const ring = (lds_u8*)dyn_lds + wave * (NBUF * SB);
  // A wave's merge rows (acc[R][D]) go into its own ring once its stream has
  // ended (its copies have all landed and been read), when they fit there; the
  // ring is refilled only after the merge's closing barrier. This keeps the
  // LDS of 16 or 32 heads per group at the ring's size.
  constexpr bool kAlias = R * D * 4 <= NBUF * SB;
  constexpr int WS = kAlias ? NBUF * SB / 4 : R * D;  // floats between waves' rows
  __shared__ float s_acc_own[kAlias ? 1 : NW * R * D];
  float* const s_acc = kAlias ? (float*)dyn_lds : s_acc_own;
  __shared__ float s_ml[NW][R][2];

  // LDS byte offsets within a stage. Score A operand: row hl, chunk 4 kk + grp.
  uint32_t offS[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) offS[kk] = hl * 256 + (((4 * kk + grp) ^ fsw(hl)) << 4);
  // Transposing reads for O^T: lane (grp, i = hl) supplies row 4 grp + i / 4,
  // columns 16 dd + 4 (i % 4) .. +3 (chunk 2 dd + (i % 4) / 2, half i % 2).
  uint32_t offT[8];
  {
    const int row = 4 * grp + (hl >> 2);
#pragma unroll
    for (int dd = 0; dd < 8; ++dd)
      offT[dd] = row * 256 + (((2 * dd + ((hl & 3) >> 1)) ^ fsw(row)) << 4) + ((hl & 1) << 3);
  }

  auto segment = [&](int b, int g, int start, int end, SegOut so) {
  const size_t bh0 = (size_t)b * p.H + g * R;

  // Score B operand of block nb: q~[h][32 kk + 8 grp .. +7] for h = 16 nb + hl
  // when h < R, zero otherwise.
  bf16x8_t qf[NB][4];
  const T* __restrict__ qp = reinterpret_cast<const T*>(p.q);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      u32x4 x = u32x4{0u, 0u, 0u, 0u};
      if (16 * nb + hl < R)
        x = *reinterpret_cast<const u32x4*>(qp + ((bh0 + 16 * nb + hl) * D + 32 * kk + 8 * grp));
      qf[nb][kk] = __builtin_bit_cast(bf16x8_t, x);
    }
  float m[NB], lsum[NB];
  f32x4_t acc[NB][8];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m[nb] = -INFINITY;
    lsum[nb] = 0.f;
#pragma unroll
    for (int dd = 0; dd < 8; ++dd) acc[nb][dd] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  auto ready = [&]() {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) asm volatile("" ::"v"(qf[nb][kk]));
  };

  // Rows at or past vend are masked: the segment's end, or the new row's
  // position while the cached rows stream when the step appends.
  int vend = end;
  auto consume = [&](const lds_u8* stage, int t0, bool blk_ok) {
    if (!blk_ok) return;  // uniform: a block outside the cache contributes nothing
    const lds_u8* ks = KEYS ? stage + TB : stage;
    f32x4_t sc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) sc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const bf16x8_t a =
          *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(ks + offS[kk]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        sc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[nb][kk], sc[nb], 0, 0, 0);
    }
    s16x4 pf[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float s4[4];
      float tmax = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float x = sc[nb][i] * p.scale_log2;
        if (t0 + 4 * grp + i >= vend) x = -INFINITY;
        s4[i] = x;
        tmax = fmaxf(tmax, x);
      }
      if (__builtin_amdgcn_ballot_w64(tmax > m[nb] + kLazy)) {
        // New reference for each head: the tile maximum over its four lane
        // groups, so the reference stays identical across them.
        float tm = fmaxf(tmax, __shfl_xor(tmax, 16));
        tm = fmaxf(tm, __shfl_xor(tm, 32));
        const float mn = (tm > m[nb] + kLazy) ? tm : m[nb];
        const float alpha = (m[nb] == -INFINITY) ? 0.f : fast_exp2(m[nb] - mn);
        lsum[nb] *= alpha;
#pragma unroll
        for (int dd = 0; dd < 8; ++dd) acc[nb][dd] *= alpha;
        m[nb] = mn;
      }
      const float nm = (m[nb] == -INFINITY) ? 0.f : -m[nb];
      float w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        w[i] = fast_exp2(s4[i] + nm);
        lsum[nb] += w[i];
      }
      pf[nb] = __builtin_bit_cast(
          s16x4, u32x2{pack_bf16_rne(w[0], w[1]), pack_bf16_rne(w[2], w[3])});
    }
#pragma unroll
    for (int dd = 0; dd < 8; ++dd) {
      const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(stage + offT[dd]));
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[nb][dd] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, pf[nb], acc[nb][dd], 0, 0, 0);
    }
  };

  const int pnew = KEYS ? -1 : new_row_in<PAGED>(p, b, start, end);
  if (pnew >= 0) vend = pnew;
  const u32x4 nrow = (pnew >= 0) ? load_new_row<T, D>(p, b, g, lane) : u32x4{0u, 0u, 0u, 0u};
  stream_tiles<T, D, PAGED, KEYS, NW>(p, b, g, lane, ring, start + wave * kTile, vend, fsw, ready,
                                      consume);
  if (pnew >= 0 && wave == 0) {  // the step's new row: from registers, not from the cache
    append_and_stage<T, D, PAGED>(p, b, g, pnew, nrow, ring, lane);
    vend = pnew + 1;
    consume(ring, pnew, true);
  }

  // Row sums of each head over the four lane groups (the reference is shared).
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float ls = lsum[nb];
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);
    const int h = 16 * nb + hl;
    if (h < R) {
#pragma unroll
      for (int dd = 0; dd < 8; ++dd)
#pragma unroll
        for (int i = 0; i < 4; ++i) s_acc[wave * WS + h * D + 16 * dd + 4 * grp + i] = acc[nb][dd][i];
      if (grp == 0) {
        s_ml[wave][h][0] = m[nb];
        s_ml[wave][h][1] = ls;
      }
    }
  }
  merge_waves<T, D, R, NW, WS>(p, s_acc, s_ml, bh0, so);
  };
  for_each_segment<T, D, R, PAGED, NW>(p, segment);
}

// Balanced-mode plan: tiles per sequence n_b = ceil(len_b / 16), their
// exclusive prefix sums pre[0..B], the total T = G pre[B] over all pairs and
// the tiles per workgroup ceil(T / nwg). One workgroup scans the sequences in
// blocks of 1024. It runs for more than kWavePlanMax sequences only.
__global__ __launch_bounds__(1024) void decode_plan_kernel(DecodeParams p) {
  __shared__ int s_scan[1024];
  __shared__ int s_carry;
  const int t = threadIdx.x;
  int* pre = p.plan + 2;
  const int cap = p.paged ? (p.max_blocks << p.block_shift) : p.L_max;
  if (t == 0) s_carry = 0;
  __syncthreads();
  for (int b0 = 0; b0 < p.B; b0 += 1024) {
    const int b = b0 + t;
    const int n = b < p.B ? (decode_rows(p, b, cap) + kTile - 1) / kTile : 0;
    s_scan[t] = n;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
      const int v = t >= off ? s_scan[t - off] : 0;
      __syncthreads();
      s_scan[t] += v;
      __syncthreads();
    }
    const int carry = s_carry;
    if (b < p.B) pre[b] = carry + s_scan[t] - n;
    __syncthreads();
    if (t == 1023) s_carry = carry + s_scan[1023];
    __syncthreads();
  }
  if (t == 0) {
    const int total = p.G * s_carry;  // the host bounds this below 2^30
    pre[p.B] = s_carry;
    p.plan[0] = total;
    p.plan[1] = total > 0 ? (total + p.nwg - 1) / p.nwg : 1;
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
  const int len = decode_rows(p, b, cap);
  int ns;                      // partials of this head
  const float* part;           // its first partial row
  size_t stride = D + 2;       // floats between consecutive partial rows
  if (!p.balanced) {
    ns = (len + p.chunk - 1) / p.chunk;
    part = p.part + (size_t)bh * p.S * (D + 2);
  } else {
    // The workgroups that covered pair (b, g) wrote partials pair + w for w in
    // [first, last]; a pair inside one workgroup was stored directly.
    int per, preb, n;
    if (p.B <= kWavePlanMax) {  // no plan kernel ran: the same plan from the lengths
      const LanePlan lp = lane_plan(p, cap);
      const int total = p.G * lp.sum;
      per = total > 0 ? (total + p.nwg - 1) / p.nwg : 1;
      preb = __builtin_amdgcn_readlane(lp.pre, b);
      n = __builtin_amdgcn_readlane(lp.n, b);
    } else {
      const int* pre = p.plan + 2;
      per = p.plan[1];
      preb = pre[b];
      n = pre[b + 1] - pre[b];
    }
    const int h = bh % p.H, g = h / p.R, r = h % p.R;
    const int tp = p.G * preb + g * n;
    const int first = n > 0 ? tp / per : 0;
    const int last = n > 0 ? (tp + n - 1) / per : -1;
    if (n > 0 && first == last) return;
    ns = last - first + 1;
    part = p.part + ((size_t)(b * p.G + g + first) * p.R + r) * (D + 2);
    stride = (size_t)p.R * (D + 2);
  }
  if (ns == 0) {
    if (t < D) store_out<T>(p.out, (size_t)bh * D + t, 0.f);
    return;
  }
  float mloc = -INFINITY;
  for (int k = t; k < ns; k += 256) mloc = fmaxf(mloc, part[k * stride + D]);
  for (int sh = 32; sh > 0; sh >>= 1) mloc = fmaxf(mloc, __shfl_xor(mloc, sh));
  if ((t & 63) == 0) s_red[t >> 6] = mloc;
  __syncthreads();
  const float M = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
  const float Ms = (M == -INFINITY) ? 0.f : M;
  __syncthreads();
  float lloc = 0.f;
  for (int k = t; k < ns; k += 256) {
    const float w = fast_exp2(part[k * stride + D] - Ms);
    s_w[k] = w;
    lloc = fmaf(part[k * stride + D + 1], w, lloc);
  }
  for (int sh = 32; sh > 0; sh >>= 1) lloc += __shfl_xor(lloc, sh);
  if ((t & 63) == 0) s_red[t >> 6] = lloc;
  __syncthreads();
  const float L = s_red[0] + s_red[1] + s_red[2] + s_red[3];
  const int c = t % D, sub = t / D;
  float a = 0.f;
#pragma unroll 4
  for (int k = sub; k < ns; k += SUB) a = fmaf(part[k * stride + c], s_w[k], a);
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
  const dim3 grid = p.balanced ? dim3(p.nwg) : dim3(p.S, p.G, p.B);
  if (p.balanced && p.B > kWavePlanMax) {
    hipLaunchKernelGGL(decode_plan_kernel, dim3(1), dim3(1024), 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (p.ev_start) {
    hipError_t e = hipEventRecord(p.ev_start, st);
    if (e != hipSuccess) return e;
  }
  // Grouped heads over a 128-wide bf16 cache run on the matrix cores.
  constexpr bool kMfma = sizeof(T) == 2 && D == 128 && R >= 2;
  constexpr int lds = Ring<T, D, KEYS, NW>::BYTES;
  static_assert(lds + NW * R * (D + 2) * 4 <= 160 * 1024, "LDS budget");
  const void* kern;
  if constexpr (kMfma)
    kern = reinterpret_cast<const void*>(decode_mfma_kernel<R, PAGED, KEYS, NW>);
  else
    kern = reinterpret_cast<const void*>(decode_partial_kernel<T, D, R, PAGED, KEYS, NW>);
  if (lds > 65536) {
    static std::atomic<uint32_t> done{0};
    hipError_t a = set_max_lds(kern, lds, done);
    if (a != hipSuccess) return a;
  }
  if constexpr (kMfma)
    hipLaunchKernelGGL((decode_mfma_kernel<R, PAGED, KEYS, NW>), grid, dim3(NW * 64), lds, st, p);
  else
    hipLaunchKernelGGL((decode_partial_kernel<T, D, R, PAGED, KEYS, NW>), grid, dim3(NW * 64), lds,
                       st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.ev_stop) {
    e = hipEventRecord(p.ev_stop, st);
    if (e != hipSuccess) return e;
  }
  if (p.balanced || p.S > 1) {
    hipLaunchKernelGGL((decode_combine_kernel<T, D>), dim3(p.B * p.H), dim3(256), 0, st, p);
    e = hipGetLastError();
  }
  return e;
}

template <typename T, int D, int R>
hipError_t pick_layout(const DecodeParams& p, hipStream_t st) {
  constexpr int NW = 4;  // waves per workgroup
  const bool keys = p.kdata != nullptr;
  if (p.paged)
    return keys ? launch_t<T, D, R, true, true, NW>(p, st) : launch_t<T, D, R, true, false, NW>(p, st);
  return keys ? launch_t<T, D, R, false, true, NW>(p, st) : launch_t<T, D, R, false, false, NW>(p, st);
}

template <typename T, int D>
hipError_t pick_r(const DecodeParams& p, hipStream_t st) {
  switch (p.R) {
    case 1: return pick_layout<T, D, 1>(p, st);
    case 2: return pick_layout<T, D, 2>(p, st);
    case 3: return pick_layout<T, D, 3>(p, st);
    case 4: return pick_layout<T, D, 4>(p, st);
    case 5: return pick_layout<T, D, 5>(p, st);
    case 6: return pick_layout<T, D, 6>(p, st);
    case 7: return pick_layout<T, D, 7>(p, st);
    case 8: return pick_layout<T, D, 8>(p, st);
    case 16:
    case 32:
      // 16 or 32 heads per group: bf16, 128-wide rows only (the matrix-core consumer).
      if constexpr (sizeof(T) == 2 && D == 128)
        return p.R == 16 ? pick_layout<T, D, 16>(p, st) : pick_layout<T, D, 32>(p, st);
      else return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, hipStream_t st) {
  if (!p.balanced && p.S > kMaxSplits) return hipErrorInvalidValue;
  if (p.balanced && (p.nwg < 1 || p.nwg > kMaxSplits || p.plan == nullptr)) return hipErrorInvalidValue;
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
