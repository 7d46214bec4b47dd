// Causal (or full) keyless attention for the bf16 prefill (Eq. 2 with the score
// of Eq. 4): O_h = softmax(tau * Q~_h V_g^T) V_g, where the value tile is both
// the "key" of the score and the value of the weighted sum. Unmasked, with the
// values taken from another sequence of Nk rows, it is the cross-attention of
// Eq. 14.
//
// A workgroup (4 waves) owns 4 * 16 * QB query rows of one head; each wave owns
// 16 * QB rows and keeps their routed-query fragments in registers. Value tiles of 64 rows
// move from memory straight into LDS (global_load_lds, 16 bytes per lane), one
// copy per tile, three tiles in flight. With v_mfma_f32_16x16x32_bf16:
//   S^T = V Q~^T     A operand = value rows (ds_read_b128 of the row-major tile)
//   O^T += V^T P^T   A operand = value columns, read from the same row-major tile
//                    with ds_read_b64_tr_b16 (each 16-lane group transposes a
//                    4-row x 16-column block into 4 rows of one column per lane)
// Computing S^T leaves each lane holding scores of one query row, so the online
// softmax needs two cross-lane steps per row, and the score registers become the
// B operand of the second product directly. The MFMA reduction order over a
// 32-row step is free as long as both operands agree; here lane group g covers
// rows 4g..4g+3 and 16+4g..16+4g+3 of the step.
// The tile's 16-byte chunks are XOR-swizzled per row so that both the score
// reads (16 rows, one chunk) and the transposed reads (8 rows, two chunks per
// pass) hit distinct LDS banks. Causal work grows with the query tile, so the
// last tiles are scheduled first, for all heads before any lighter tile.
// Causal calls take QB = 3 (192 query rows per workgroup: every LDS fragment
// read feeds three products); unmasked calls take QB = 2 (128 rows), whose finer
// grid fills the chip in whole waves of workgroups on common shapes (1024
// attending rows: 8 tiles per head instead of 5 1/3). Each output row is
// computed the same way in both: the results are bit-identical.

#include <type_traits>

#include "attn_tile.h"
#include "kl_device.h"
#include "kl_internal.h"

namespace kl {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) unsigned char lds_u8;

constexpr int BKV = 64;     // value rows per tile
constexpr int NSTAGE = 3;   // value tiles in flight (the tile loop is unrolled by 3)
static_assert(NSTAGE == 3, "the tile loop below calls process once per stage, three per pass");
constexpr int kThreads = 256;
// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

// max(a, b, c); written for the compiler (not as inline assembly, which would
// hide a read of a fresh MFMA result from its hazard checks), which forms
// v_max3_f32 since this file is built without NaN semantics.
__device__ __forceinline__ float max3(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }

template <int D>
using Tile = AttnTile<D, BKV>;

// QB: 16-row query blocks per wave.
template <int D, int QB>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(AttnParams p) {
  constexpr int WQ = 16 * QB;  // query rows per wave
  constexpr int BQ = 4 * WQ;   // query rows per workgroup
  using T = Tile<D>;
  constexpr int KS = D / 32;  // MFMA k-steps over d_head for S^T
  constexpr int DB = D / 16;  // 16-wide column blocks of the output
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];  // NSTAGE tiles

  const int ntq = (p.N + BQ - 1) / BQ;
  // Heads vary fastest in the grid: workgroups are dispatched in linear-id
  // order, so every head's heaviest (causal) query tile starts first, and
  // workgroup i runs on XCD i % 8, so each XCD keeps whole heads' values in
  // its own L2.
  const int qt = p.causal ? (ntq - 1 - (int)blockIdx.y) : (int)blockIdx.y;
  const int h = blockIdx.x, b = blockIdx.z;
  const int g = h / (p.H / p.G);
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int fr = lane & 15, grp = lane >> 4;
  const int q0 = qt * BQ + wave * WQ;  // this wave's first query row

  const uint16_t* __restrict__ Q = reinterpret_cast<const uint16_t*>(p.q);

  f32x4_t o[DB][QB];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) o[i][qb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // Row sums of the weights, from the same MFMA with an all-ones A operand: every
  // row of the product is the column sum of P^T, i.e. the weight sum per query.
  f32x4_t osum[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) osum[qb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const bf16x8_t ones = __builtin_bit_cast(
      bf16x8_t, u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
  float m[QB];  // reference exponent per query block; set by the first tile
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) m[qb] = 0.f;

  // Tile copies: wave copy c of this wave fills tile rows 4 (c * 4 + wave) ..
  // + 3; lane L lands at row + L / CHUNKS, physical chunk L % CHUNKS. Rows past
  // the end are clamped: their scores are masked, so they carry no weight.
  const unsigned char* gV = reinterpret_cast<const unsigned char*>(p.v);
  constexpr int ROWS_PER_COPY = 1024 / T::ROW;
  // The copy's source is a wave-uniform base (first row of the group, clamped)
  // plus a per-lane offset (row within the group, clamped, and chunk).
  uint32_t col_off[T::COPIES];  // bytes: group g's columns plus the logical chunk (+ the lane's row below)
#pragma unroll
  for (int c = 0; c < T::COPIES; ++c) {
    const int r = (c * 4 + wave) * ROWS_PER_COPY + lane / T::CHUNKS;
    const int pc = lane % T::CHUNKS;
    int lc = pc;
    // invert the swizzle: logical chunk whose physical position is pc
#pragma unroll
    for (int x = 0; x < T::CHUNKS; ++x)
      if (T::swz(r, x) == pc) lc = x;
    col_off[c] = (uint32_t)(((size_t)g * D + lc * 8) * 2);
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)smem;
  const size_t row_bytes = (size_t)p.v_stride * 2;
  const uint32_t lane_row = (uint32_t)(lane / T::CHUNKS) * (uint32_t)row_bytes;
#pragma unroll
  for (int c = 0; c < T::COPIES; ++c) col_off[c] += lane_row;  // now the whole per-lane offset
  auto issue = [&](int jt, const int stage) {
    const int j0 = jt * BKV;
    if (j0 + BKV <= p.Nk) {
      // Every row of the tile exists: one base per tile, per-copy steps uniform.
      const unsigned char* tb = gV + ((size_t)b * p.Nk + j0) * row_bytes;
#pragma unroll
      for (int c = 0; c < T::COPIES; ++c)
        copy_to_lds(tb + (size_t)((c * 4 + wave) * ROWS_PER_COPY) * row_bytes, col_off[c],
                    lds0 + stage * T::BYTES + (c * 4 + wave) * 1024);
    } else {
#pragma unroll
      for (int c = 0; c < T::COPIES; ++c) {
        const int r0 = j0 + (c * 4 + wave) * ROWS_PER_COPY;  // uniform
        const int r0c = min(r0, p.Nk - 1);
        const int rl = min(r0 + lane / T::CHUNKS, p.Nk - 1) - r0c;  // 0 .. ROWS_PER_COPY - 1
        const unsigned char* base = gV + ((size_t)b * p.Nk + r0c) * row_bytes;
        copy_to_lds(base, (uint32_t)(rl * row_bytes) + col_off[c] - lane_row,
                    lds0 + stage * T::BYTES + (c * 4 + wave) * 1024);
      }
    }
  };

  // Per-lane LDS byte offsets inside a tile, formed at each use from two
  // registers per read kind (score operand: row fr, chunk 4 ks + grp, + 16 kb
  // rows; transposed operand: row 4 grp + fr / 4, columns 16 db + 4 (fr % 4)).
  // The swizzle of a row depends only on the lane here, so the block, step and
  // stage offsets are immediates. As a table of KS + DB registers they pushed
  // the kernel past its register budget, and the spilled entry's reload inside
  // the tile loop came with a wait for every load in flight, the next tiles'
  // copies included.
  FragOffsets<D> fo(fr, grp);
  fo.sbase += (int)lds0;  // absolute LDS addresses: the tile's own offset is an immediate
  fo.tbase += (int)lds0;

  const int last_row = p.causal ? min(qt * BQ + BQ, p.Nk) : p.Nk;
  const int ntiles = (last_row + BKV - 1) / BKV;
#pragma unroll
  for (int s = 0; s < NSTAGE - 1; ++s)
    if (s < ntiles) issue(s, s);

  // Routed-query fragments (B operand of S^T), loaded after the first value
  // tiles are requested so that the two latencies overlap (light causal tiles,
  // which run last, are dominated by them): query row q0 + 16 qb + fr,
  // columns 32 ks + 8 grp .. + 7, multiplied by c = scale * log2(e) and rounded
  // to bf16 once, so the products come out in exponent (log2) units. Rows past
  // the end are clamped (never stored).
  const float c = p.scale_log2;
  bf16x8_t qf[QB][KS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qq = min(q0 + qb * 16 + fr, p.N - 1);
    const uint16_t* src = Q + ((size_t)b * p.N + qq) * p.q_stride + (size_t)h * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(src + ks * 32);
      u32x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = pack2(__uint_as_float(raw[j] << 16) * c, __uint_as_float(raw[j] & 0xFFFF0000u) * c);
      qf[qb][ks] = __builtin_bit_cast(bf16x8_t, w);
    }
  }


  // One value tile. Scores come out of the MFMA already shifted by the
  // reference: the accumulation starts from -m (in log2 units, as q carries c).
  // The reference moves lazily, only when a score exceeds it by more than 2^8,
  // which keeps every weight below 256 and skips the rescale of O on most
  // tiles; the first tile (row 0 is always unmasked) sets it exactly.
  auto process = [&](const int jt, auto stage_tag, auto first_tag) {
    constexpr int STAGE = decltype(stage_tag)::value;
    constexpr bool FIRST = decltype(first_tag)::value;
    // Tile jt has landed once at most the copies of the later issued tiles
    // (jt + 1 .. jt + NSTAGE - 2) remain.
    if (jt + 1 < ntiles) KL_WAIT_VMCNT((NSTAGE - 2) * T::COPIES);
    else KL_WAIT_VMCNT(0);
    // The copies issued below refill the stage of tile jt - 1: every wave's LDS
    // reads of it must have returned before the barrier (the barrier itself does
    // not wait for outstanding LDS reads).
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __syncthreads();
    if (jt + NSTAGE - 1 < ntiles) issue(jt + NSTAGE - 1, (STAGE + NSTAGE - 1) % NSTAGE);
    const int j0 = jt * BKV;
    // Skip tiles entirely above the diagonal for this wave (never the first),
    // and every tile for a wave whose rows all lie past the end (a ragged last
    // query tile): such a wave still copies and meets the barriers.
    if (q0 >= p.N || (!FIRST && p.causal && j0 > q0 + WQ - 1)) return;
    // fo gives absolute LDS addresses in stage 0; this stage's offset is an immediate.
    constexpr uint32_t tile = STAGE * T::BYTES;
    auto at = [](uint32_t a) { return (const lds_u8*)(uintptr_t)a; };

    // S^T[kv][q] - m[q] for kv blocks kb (16 rows) and query blocks qb.
    f32x4_t init[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
      init[qb] = FIRST ? f32x4_t{0.f, 0.f, 0.f, 0.f} : f32x4_t{-m[qb], -m[qb], -m[qb], -m[qb]};
    // The fragments of block kb + 1 are read while the products of block kb
    // run (two register sets); the schedule below pins that order, since the
    // compiler otherwise issues each read just before its use and waits for it.
    f32x4_t sc[4][QB];
    {
      int offS[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) offS[ks] = fo.s(ks);
      bf16x8_t sa[2][KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sa[0][ks] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(at(tile + offS[ks]));
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        if (kb + 1 < 4) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            sa[(kb + 1) & 1][ks] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
                at(tile + offS[ks] + (kb + 1) * 16 * T::ROW));
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            sc[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sa[kb & 1][ks], qf[qb][ks],
                                                                 ks == 0 ? init[qb] : sc[kb][qb], 0, 0, 0);
      }
      // Groups in order: the reads of block 0, then (reads of block kb + 1,
      // products of block kb) for kb < 3, then the products of block 3.
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, KS, 0);
#pragma unroll
      for (int kb = 0; kb < 3; ++kb) {
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, KS, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, KS * QB, 0);
      }
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, KS * QB, 0);
    }
    // Lane holds scores of query q0 + 16 qb + fr against rows j0 + 16 kb + 4 grp + r.
    if ((p.causal && j0 + BKV - 1 > q0) || (j0 + BKV > p.Nk)) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int q = q0 + qb * 16 + fr;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int kv = j0 + kb * 16 + grp * 4 + r;
            if (kv >= p.Nk || (p.causal && kv > q)) sc[kb][qb][r] = -INFINITY;
          }
      }
    }
    float lm[QB];  // this lane's maximum per query block (16 scores: 8 three-way maxima)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float v = max3(sc[0][qb][0], sc[0][qb][1], sc[0][qb][2]);
      v = max3(v, sc[0][qb][3], sc[1][qb][0]);
      v = max3(v, sc[1][qb][1], sc[1][qb][2]);
      v = max3(v, sc[1][qb][3], sc[2][qb][0]);
      v = max3(v, sc[2][qb][1], sc[2][qb][2]);
      v = max3(v, sc[2][qb][3], sc[3][qb][0]);
      v = max3(v, sc[3][qb][1], sc[3][qb][2]);
      lm[qb] = fmaxf(v, sc[3][qb][3]);
    }
    bool grow = FIRST;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) grow |= lm[qb] > 8.f;
    if (FIRST || __builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        // Tile maximum of each query over its four lane groups.
        float t = fmaxf(lm[qb], __shfl_xor(lm[qb], 16));
        t = fmaxf(t, __shfl_xor(t, 32));
        const float d = FIRST ? t : (t > 8.f ? t : 0.f);
        m[qb] += d;
        if (!FIRST) {
          const float alpha = fast_exp2(-d);
#pragma unroll
          for (int i = 0; i < DB; ++i) o[i][qb] *= alpha;
          osum[qb] *= alpha;
        }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) sc[kb][qb] -= d;
      }
    }
    // Weights and P^T fragments of one 32-row k-step (rows 32 ks + {4 grp ..
    // 4 grp + 3, 16 + 4 grp ..}), for every query block.
    bf16x8_t pf[QB][2];
    auto weights = [&](const int ks) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        u32x4 w;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          f32x4_t& x = sc[2 * ks + h][qb];
          x[0] = fast_exp2(x[0]);
          x[1] = fast_exp2(x[1]);
          x[2] = fast_exp2(x[2]);
          x[3] = fast_exp2(x[3]);
          w[2 * h] = pack2(x[0], x[1]);
          w[2 * h + 1] = pack2(x[2], x[3]);
        }
        pf[qb][ks] = __builtin_bit_cast(bf16x8_t, w);
      }
    };
    // O^T[d][q] += V^T P^T over one k-step: the transposed read hands lane fr
    // the 4 rows of column 16 db + fr (rows 32 ks + 4 grp .., and 16 further
    // for the high half); the all-ones operand adds the weight sums. All reads
    // of the k-step are issued ahead of its products.
    int offT[DB];
    auto pv = [&](const int ks) {
      bf16x8_t av[DB];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const lds_u8* src = at(tile + offT[db] + ks * 32 * T::ROW);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(src));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(src + 16 * T::ROW));
        av[db] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          o[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[db], pf[qb][ks], o[db][qb], 0, 0, 0);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        osum[qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[qb][ks], osum[qb], 0, 0, 0);
    };
    weights(0);
    weights(1);
#pragma unroll
    for (int db = 0; db < DB; ++db) offT[db] = fo.t(db);
    pv(0);
    pv(1);
  };

  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  process(0, I0{}, std::true_type{});  // tile 0 is never above the diagonal
  if (1 < ntiles) process(1, I1{}, std::false_type{});
  if (2 < ntiles) process(2, I2{}, std::false_type{});
  for (int jt = NSTAGE; jt < ntiles; jt += NSTAGE) {
    process(jt, I0{}, std::false_type{});
    if (jt + 1 < ntiles) process(jt + 1, I1{}, std::false_type{});
    if (jt + 2 < ntiles) process(jt + 2, I2{}, std::false_type{});
  }

  // Normalise and store: lane holds O[q][16 db + 4 grp + r] for its query rows.
  uint16_t* __restrict__ O = reinterpret_cast<uint16_t*>(p.out);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l = osum[qb][0];
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const int q = q0 + qb * 16 + fr;
    if (p.lse && q < p.N && grp == 0)  // scores are in log2 units relative to m
      p.lse[((size_t)b * p.H + h) * p.N + q] = (m[qb] + __log2f(l)) * 0.69314718055994531f;
    if (p.out_f32 && q < p.N) {
      float* dst = p.out_f32 + (((size_t)b * p.N + q) * p.H + h) * D + grp * 4;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<f32x4_t*>(dst + db * 16) =
            f32x4_t{o[db][qb][0] * inv, o[db][qb][1] * inv, o[db][qb][2] * inv, o[db][qb][3] * inv};
    }
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

template <int D, int QB>
hipError_t launch_attn_qb(const AttnParams& p, hipStream_t st) {
  constexpr int BQ = 4 * 16 * QB;
  dim3 grid(p.H, (p.N + BQ - 1) / BQ, p.B);
  hipLaunchKernelGGL((attn_bf16_kernel<D, QB>), grid, dim3(kThreads), NSTAGE * Tile<D>::BYTES, st, p);
  return hipGetLastError();
}

template <int D>
hipError_t launch_attn(const AttnParams& p, hipStream_t st) {
  return p.causal ? launch_attn_qb<D, 3>(p, st) : launch_attn_qb<D, 2>(p, st);
}

}  // namespace

bool attn_bf16_supported(const AttnParams& p) {
  // Strides keep 16-byte alignment; a copy's per-lane offset spans at most 8
  // value rows and must fit in 32 bits.
  return p.dtype == KL_BF16 && (p.D == 64 || p.D == 128) && p.q_stride % 8 == 0 &&
         p.v_stride % 8 == 0 && p.o_stride % 8 == 0 && (size_t)p.v_stride * 2 * 8 < (1u << 31);
}

hipError_t launch_prefill_attention(const AttnParams& p, hipStream_t st) {
  if (p.N == 0 || p.B == 0) return hipSuccess;
  if (p.Nk <= 0 || (p.causal && p.Nk != p.N)) return hipErrorInvalidValue;
  if (p.D == 128) return launch_attn<128>(p, st);
  if (p.D == 64) return launch_attn<64>(p, st);
  return hipErrorInvalidValue;
}

}  // namespace kl
