// Backward pass of keyless attention (Section 2.3): given dL/dO, the gradients
// of the routed queries and of the values. Per batch b and head h (group g):
//   P   = exp(tau Q~ V^T - lse)        (the forward's weights, from its log-sum-exp)
//   dP  = dO V^T
//   dS  = P * (dP - Dd),  Dd = rowsum(P * dP) = rowsum(dO * O)   (softmax backward)
//   dQ~ = tau dS V
//   dV  = P^T dO + tau dS^T Q~        (retrieval and routing terms of Eq. 6)
// The value tile is read once per product it enters, exactly as in the
// forward: as the score operand and as the retrieved values (dQ~ kernel), and
// the value gradient collects both of its roles in the same accumulators.
//
// bf16: bwd_dq_kernel (one workgroup per 128-row query tile and head; value
// tiles stream through LDS as in the forward, queries and dO stay in
// registers; Dd = rowsum(dO * O) from the forward's fp32 output when the
// caller kept it, formed in the kernel's prologue, else a first sweep forms
// it as rowsum(P * dP) in fp32, since rowsum(dO * O) over the bf16-rounded
// output would put that rounding into every dP - Dd) and then bwd_dv_kernel
// (one workgroup per 192-row value tile and value group; query and dO tiles of
// every head of the group stream through LDS, the values stay in registers).
// fp32 (and shapes the matrix-core kernels do not take): bwd_prep_kernel (Dd
// from the fp32 output, else from the output) and two vector-ALU kernels. No
// atomics: every output element is written once, by one lane.
//
// bf16 runs on v_mfma_f32_16x16x32_bf16 with the forward's operand layouts:
// scores come out with one query per lane (S^T = V Q~^T) in the dQ~ kernel and
// one value row per lane (S = Q~ V^T) in the dV kernel, and in both the weights
// feed the next product as its B operand without a transpose; the transposed
// A operands come from ds_read_b64_tr_b16 on the row-major tiles. fp32 runs
// VALU kernels of the same structure.

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

constexpr int kThreads = 256;
constexpr int kTileRows = 64;   // rows per staged tile
// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;
constexpr float kLog2e = 1.4426950408889634f;

// One 4-byte-per-lane copy from global memory straight into LDS
// (global_load_lds_dword): lane L's word lands at lds + 4 L; otherwise as
// copy_to_lds (counted by vmcnt, not by the compiler).
__device__ __forceinline__ void copy_dword_to_lds(const void* gbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(gbase), "s"(lds)
               : "memory", "m0");
}

template <typename T>
__device__ __forceinline__ float ldx(const T* p, size_t i) {
  if constexpr (sizeof(T) == 2) return __uint_as_float((uint32_t)p[i] << 16);
  else return p[i];
}
template <typename T>
__device__ __forceinline__ void stx(T* p, size_t i, float v) {
  if constexpr (sizeof(T) == 2) p[i] = __builtin_bit_cast(uint16_t, (__bf16)v);
  else p[i] = v;
}

// Dd[b, h, q] = sum_d dO[b, q, h, d] O[b, q, h, d] for the vector-ALU kernels;
// 16 lanes per row. O is the forward's fp32 output when given (TO = float, row
// stride H D), else `out`.
template <typename TO, typename T, int D>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdParams p) {
  const long rows = (long)p.B * p.N * p.H;
  const long row = (long)blockIdx.x * 16 + threadIdx.x / 16;
  const int j = threadIdx.x % 16;
  float s = 0.f;
  int b = 0, q = 0, h = 0;
  if (row < rows) {
    h = (int)(row % p.H);
    const long bq = row / p.H;
    b = (int)(bq / p.N);
    q = (int)(bq % p.N);
    const TO* o = p.out_f32 ? reinterpret_cast<const TO*>(p.out_f32) + ((size_t)bq * p.H + h) * D
                            : reinterpret_cast<const TO*>(p.out) + (size_t)bq * p.o_stride + (size_t)h * D;
    const T* g = reinterpret_cast<const T*>(p.dout) + (size_t)bq * p.o_stride + (size_t)h * D;
#pragma unroll
    for (int c = j; c < D; c += 16) s = fmaf(ldx(o, c), ldx(g, c), s);
  }
  s += __shfl_xor(s, 8);
  s += __shfl_xor(s, 4);
  s += __shfl_xor(s, 2);
  s += __shfl_xor(s, 1);
  if (row < rows && j == 0) p.Dd[((size_t)b * p.H + h) * p.N + q] = s;
}

// ---------------------------------------------------------------------------
// bf16, matrix cores
// ---------------------------------------------------------------------------

constexpr int QBD = 2;                 // 16-row query blocks per wave (dQ~ kernel)
constexpr int BQD = 4 * 16 * QBD;      // query rows per workgroup
constexpr int NSTAGE = 3;              // value tiles in flight (dQ~ kernel)
static_assert(NSTAGE >= 2, "the dQ~ kernel's ring needs two stages");
constexpr int KVB = 3;                 // 16-row value blocks per wave (dV kernel)
constexpr int BKVD = 4 * 16 * KVB;     // value rows per workgroup

// Direct-to-LDS copy of rows [row0, row0 + 64) (clamped to n_rows - 1) of a
// row-major bf16 matrix, columns [col, col + D), into an AttnTile<D, 64>. Wave
// copy c fills tile rows 4 (c * 4 + wave) .. + 3 (D = 128) or 8 (..) .. + 7
// (D = 64); lane L lands at physical chunk L % CHUNKS of its row and fetches
// the logical chunk that the swizzle puts there.
template <int D>
struct TileCopier {
  using TL = AttnTile<D, kTileRows>;
  static constexpr int ROWS_PER_COPY = 1024 / TL::ROW;
  uint32_t chunk_off[TL::COPIES];  // bytes of the fetched logical chunk
  __device__ __forceinline__ explicit TileCopier(int wave, int lane) {
#pragma unroll
    for (int c = 0; c < TL::COPIES; ++c) {
      const int r = (c * 4 + wave) * ROWS_PER_COPY + lane / TL::CHUNKS;
      const int pc = lane % TL::CHUNKS;
      int lc = pc;
#pragma unroll
      for (int x = 0; x < TL::CHUNKS; ++x)
        if (TL::swz(r, x) == pc) lc = x;
      chunk_off[c] = (uint32_t)(lc * 16);
    }
  }
  __device__ __forceinline__ void issue(const unsigned char* g, size_t row_bytes, uint32_t col_bytes,
                                        int row0, int n_rows, int wave, int lane,
                                        uint32_t lds) const {
#pragma unroll
    for (int c = 0; c < TL::COPIES; ++c) {
      const int r0 = row0 + (c * 4 + wave) * ROWS_PER_COPY;  // uniform
      const int r0c = min(r0, n_rows - 1);
      const int rl = min(r0 + lane / TL::CHUNKS, n_rows - 1) - r0c;
      copy_to_lds(g + (size_t)r0c * row_bytes, (uint32_t)(rl * row_bytes) + col_bytes + chunk_off[c],
                  lds + (c * 4 + wave) * 1024);
    }
  }
};

// dQ~ for 128 query rows of one head. Mirrors the forward kernel: S^T = V Q~^T
// and dP^T = V dO^T share each value-row fragment read; dS^T feeds
// dQ~^T += V^T dS^T as the B operand.
// SWEEP0: Dd is formed here in a first sweep (no fp32 output); else the
// prologue forms it from the fp32 output and one sweep does. Either way it is
// written for the dV kernel.
template <int D, bool SWEEP0>
__global__ __launch_bounds__(kThreads, 2) void bwd_dq_kernel(BwdParams p) {
  using TL = AttnTile<D, kTileRows>;
  constexpr int KS = D / 32, DB = D / 16;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  const int ntq = (p.N + BQD - 1) / BQD;
  // Heads fastest in the grid (heaviest causal tiles of every head first; each
  // XCD, which runs workgroups i with i % 8 fixed, keeps whole heads).
  const int qt = p.causal ? (ntq - 1 - (int)blockIdx.y) : (int)blockIdx.y;
  const int h = blockIdx.x, b = blockIdx.z;
  const int g = h / (p.H / p.G);
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int fr = lane & 15, grp = lane >> 4;
  const int q0 = qt * BQD + wave * 16 * QBD;
  const uint16_t* __restrict__ Q = reinterpret_cast<const uint16_t*>(p.q);
  const uint16_t* __restrict__ dO = reinterpret_cast<const uint16_t*>(p.dout);
  const float c = p.scale_log2;

  // B operands: query row q0 + 16 qb + fr, columns 32 ks + 8 grp .. + 7; the
  // routed query multiplied by c and rounded to bf16 as in the forward.
  bf16x8_t qf[QBD][KS], df[QBD][KS];
  // One sweep: the score and dP accumulators start from -lse (log2 units) and
  // -Dd, both per query (one per lane column), so P = 2^S and dS = P dP come
  // straight out of the products. The two-sweep form, at its register limit,
  // subtracts them (lse2, dd) instead.
  f32x4_t nlse[QBD], ndd[QBD];
  float lse2[QBD], dd[QBD];
#pragma unroll
  for (int qb = 0; qb < QBD; ++qb) {
    const int qq = min(q0 + qb * 16 + fr, p.N - 1);
    const uint16_t* sq = Q + ((size_t)b * p.N + qq) * p.q_stride + (size_t)h * D + grp * 8;
    const uint16_t* sd = dO + ((size_t)b * p.N + qq) * p.o_stride + (size_t)h * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(sq + ks * 32);
      u32x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = pack2(__uint_as_float(raw[j] << 16) * c, __uint_as_float(raw[j] & 0xFFFF0000u) * c);
      qf[qb][ks] = __builtin_bit_cast(bf16x8_t, w);
      df[qb][ks] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(sd + ks * 32));
    }
    const float l2 = p.lse[((size_t)b * p.H + h) * p.N + qq] * kLog2e;
    if constexpr (SWEEP0) {
      lse2[qb] = l2;
      dd[qb] = 0.f;  // from the first sweep
    } else {
      // Dd = rowsum(dO * O) from the forward's fp32 output: this lane's 32
      // columns of the row (where its dO fragments are), then the 4 lane groups;
      // published for the dV kernel.
      const float* o = p.out_f32 + (((size_t)b * p.N + qq) * p.H + h) * D + grp * 8;
      float d0 = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const f32x4_t o0 = *reinterpret_cast<const f32x4_t*>(o + ks * 32);
        const f32x4_t o1 = *reinterpret_cast<const f32x4_t*>(o + ks * 32 + 4);
        const u32x4 g = __builtin_bit_cast(u32x4, df[qb][ks]);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          d0 = fmaf(__uint_as_float(g[j] << 16), o0[2 * j], d0);
          d0 = fmaf(__uint_as_float(g[j] & 0xFFFF0000u), o0[2 * j + 1], d0);
          d0 = fmaf(__uint_as_float(g[j + 2] << 16), o1[2 * j], d0);
          d0 = fmaf(__uint_as_float(g[j + 2] & 0xFFFF0000u), o1[2 * j + 1], d0);
        }
      }
      d0 += __shfl_xor(d0, 16);
      d0 += __shfl_xor(d0, 32);
      if (grp == 0 && q0 + qb * 16 + fr < p.N) p.Dd[((size_t)b * p.H + h) * p.N + qq] = d0;
      nlse[qb] = f32x4_t{-l2, -l2, -l2, -l2};
      ndd[qb] = f32x4_t{-d0, -d0, -d0, -d0};
    }
  }
  f32x4_t acc[DB][QBD];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int qb = 0; qb < QBD; ++qb) acc[i][qb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const TileCopier<D> cp(wave, lane);
  const unsigned char* gV = reinterpret_cast<const unsigned char*>(p.v);
  const size_t vrow = (size_t)p.v_stride * 2;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)smem;
  auto issue = [&](int jt, int stage) {
    cp.issue(gV + (size_t)b * p.N * vrow, vrow, (uint32_t)(g * D * 2), jt * kTileRows, p.N, wave,
             lane, lds0 + stage * TL::BYTES);
  };
  const FragOffsets<D> fo(fr, grp);
  const int last_row = p.causal ? min(qt * BQD + BQD, p.N) : p.N;
  const int ntiles = (last_row + kTileRows - 1) / kTileRows;

  // Two sweeps over the value tiles. The first forms Dd = sum_j P_ij dP_ij in
  // fp32 (the definition, rather than rowsum(dO * O) from the rounded output,
  // whose rounding the subtraction dP - Dd would amplify) and writes it for the
  // dV kernel; the second forms dS and accumulates dQ~.
  // With the forward's fp32 output, the prologue formed Dd and one sweep does.
#pragma unroll 1
  for (int sweep = SWEEP0 ? 0 : 1; sweep < 2; ++sweep) {
    if (sweep == 1) {
      // Every wave's reads of the first sweep's last stages have returned.
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __syncthreads();
    }
    // The first tiles' copy addresses are formed here, per sweep: hoisted out
    // of the sweep loop by the compiler, they were spilled, and each reload
    // came with a wait for every copy already in flight.
    int t0 = 0;
    asm volatile("" : "+s"(t0));
#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s)
      if (s < ntiles) issue(t0 + s, s);
    float dsum[QBD];
#pragma unroll
    for (int qb = 0; qb < QBD; ++qb) dsum[qb] = 0.f;

    for (int jt = 0; jt < ntiles; ++jt) {
      const int stage = jt % NSTAGE;
      // Tiles jt + 1 .. jt + NSTAGE - 2 may stay in flight (the last tile waits for all).
      if (jt + 1 < ntiles) KL_WAIT_VMCNT((NSTAGE - 2) * TL::COPIES);
      else KL_WAIT_VMCNT(0);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __syncthreads();
      if (jt + NSTAGE - 1 < ntiles) issue(jt + NSTAGE - 1, (jt + NSTAGE - 1) % NSTAGE);
      const int j0 = jt * kTileRows;
      // Above this wave's diagonal, or rows all past the end (a ragged last tile).
      if (q0 >= p.N || (p.causal && j0 > q0 + 16 * QBD - 1)) continue;
      // Fragment offsets from this tile's stage: one v_xad_u32 forms a read's
      // whole address (the row blocks are immediate offsets). The two-sweep
      // form, at its register limit, keeps them relative and adds the stage.
      const uint32_t sbase = lds0 + stage * TL::BYTES;
      const FragOffsets<D> fi = SWEEP0 ? fo : fo.at(sbase);
      const uint32_t sadd = SWEEP0 ? sbase : 0u;
      auto lds_at = [&](int a) { return (const lds_u8*)(size_t)((uint32_t)a + sadd); };

      // Tiles on this wave's diagonal or past the sequence's end mask weights
      // (one uniform test per block of weights).
      const bool edge = (p.causal && j0 + kTileRows - 1 > q0) || (j0 + kTileRows > p.N);
      // One 32-row k-step at a time (value blocks kb = 2 ks, 2 ks + 1), which
      // keeps half of the tile's scores live.
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        f32x4_t sc[2][QBD], dp[2][QBD];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int qb = 0; qb < QBD; ++qb) {
            if constexpr (SWEEP0) {
              sc[hh][qb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
              dp[hh][qb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            } else {
              sc[hh][qb] = nlse[qb];
              dp[hh][qb] = ndd[qb];
            }
          }
        // Both blocks' value fragments are read up front; the schedule puts the
        // second block's reads between the first block's products.
        bf16x8_t va[2][KS];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int kd = 0; kd < KS; ++kd)
            va[hh][kd] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(
                lds_at(fi.s(kd)) + (2 * ks + hh) * 16 * TL::ROW);
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int kd = 0; kd < KS; ++kd)
#pragma unroll
            for (int qb = 0; qb < QBD; ++qb) {
              sc[hh][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[hh][kd], qf[qb][kd], sc[hh][qb], 0, 0, 0);
              dp[hh][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[hh][kd], df[qb][kd], dp[hh][qb], 0, 0, 0);
            }
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, KS, 0);
#pragma unroll
        for (int kd = 0; kd < KS; ++kd) {
          __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2 * QBD, 0);
          __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2 * QBD * KS, 0);
        // Lane: rows j0 + 16 (2 ks + hh) + 4 grp + r of query q0 + 16 qb + fr.
        // The weights, masked on tiles at this wave's diagonal or past the
        // sequence's end; the test is uniform, taken once per k-step.
        auto weights = [&](auto masked_tag, auto use) {
          constexpr bool MASKED = decltype(masked_tag)::value;
#pragma unroll
          for (int qb = 0; qb < QBD; ++qb)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                float pr = fast_exp2(SWEEP0 ? sc[hh][qb][r] - lse2[qb] : sc[hh][qb][r]);
                if constexpr (MASKED) {
                  const int kv = j0 + (2 * ks + hh) * 16 + grp * 4 + r;
                  pr = (kv >= p.N || (p.causal && kv > q0 + qb * 16 + fr)) ? 0.f : pr;
                }
                use(qb, hh, r, pr);
              }
        };
        if (sweep == 0) {
          auto acc_dd = [&](int qb, int hh, int r, float pr) {
            dsum[qb] = fmaf(pr, dp[hh][qb][r], dsum[qb]);
          };
          if (edge) weights(std::true_type{}, acc_dd);
          else weights(std::false_type{}, acc_dd);
          continue;
        }
        // dS^T fragments of the k-step (rows 32 ks + {4 grp .., 16 + 4 grp ..}).
        float dsv[QBD][2][4];
        auto keep_ds = [&](int qb, int hh, int r, float pr) {
          dsv[qb][hh][r] = pr * (SWEEP0 ? dp[hh][qb][r] - dd[qb] : dp[hh][qb][r]);
        };
        if (edge) weights(std::true_type{}, keep_ds);
        else weights(std::false_type{}, keep_ds);
        bf16x8_t pf[QBD];
#pragma unroll
        for (int qb = 0; qb < QBD; ++qb) {
          u32x4 w;
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            w[2 * hh] = pack2(dsv[qb][hh][0], dsv[qb][hh][1]);
            w[2 * hh + 1] = pack2(dsv[qb][hh][2], dsv[qb][hh][3]);
          }
          pf[qb] = __builtin_bit_cast(bf16x8_t, w);
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const lds_u8* src = lds_at(fi.t(db)) + ks * 32 * TL::ROW;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4*)(src));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4*)(src + 16 * TL::ROW));
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
          for (int qb = 0; qb < QBD; ++qb)
            acc[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pf[qb], acc[db][qb], 0, 0, 0);
        }
      }
    }
    if (sweep == 0) {
      // Sum each query's rows over the four lane groups; publish Dd.
#pragma unroll
      for (int qb = 0; qb < QBD; ++qb) {
        float t = dsum[qb] + __shfl_xor(dsum[qb], 16);
        t += __shfl_xor(t, 32);
        dd[qb] = t;
        const int q = q0 + qb * 16 + fr;
        if (grp == 0 && q < p.N) p.Dd[((size_t)b * p.H + h) * p.N + q] = t;
      }
    }
  }

  // Lane holds dQ~^T[16 db + 4 grp + r][q]; dQ~ = tau dS V.
  uint16_t* __restrict__ out = reinterpret_cast<uint16_t*>(p.dq);
#pragma unroll
  for (int qb = 0; qb < QBD; ++qb) {
    const int q = q0 + qb * 16 + fr;
    if (q >= p.N) continue;
    uint16_t* dst = out + ((size_t)b * p.N + q) * p.dq_stride + (size_t)h * D + grp * 4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const u32x2 w{pack2(acc[db][qb][0] * p.scale, acc[db][qb][1] * p.scale),
                    pack2(acc[db][qb][2] * p.scale, acc[db][qb][3] * p.scale)};
      *reinterpret_cast<u32x2*>(dst + db * 16) = w;
    }
  }
}

// dV for 192 value rows of one group: every head of the group and every query
// tile that can see these rows stream through LDS (routed queries and dO, two
// stages); the wave's 48 value rows stay in registers as the B operand of
// S = Q~ V^T and dP = dO V^T, whose results (one value row per lane) are the B
// operands of dV^T += dO^T P + tau Q~^T dS.
template <int D>
__global__ __launch_bounds__(kThreads, 2) void bwd_dv_kernel(BwdParams p) {
  using TL = AttnTile<D, kTileRows>;
  constexpr int KS = D / 32, DB = D / 16;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  // Groups fastest in the grid, as in the dQ~ kernel (value tile 0 is the
  // heaviest under the causal mask).
  const int kvt = blockIdx.y, g = blockIdx.x, b = blockIdx.z;
  const int R = p.H / p.G;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int fr = lane & 15, grp = lane >> 4;
  const int kv0 = kvt * BKVD + wave * 16 * KVB;  // this wave's first value row
  const float c = p.scale_log2;

  // B operands: value row kv0 + 16 kb + fr, columns 32 ks + 8 grp .. + 7.
  bf16x8_t vf[KVB][KS];
  const uint16_t* __restrict__ V = reinterpret_cast<const uint16_t*>(p.v);
#pragma unroll
  for (int kb = 0; kb < KVB; ++kb) {
    const int kv = min(kv0 + kb * 16 + fr, p.N - 1);
    const uint16_t* sv = V + ((size_t)b * p.N + kv) * p.v_stride + (size_t)g * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      vf[kb][ks] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(sv + ks * 32));
  }
  f32x4_t acc[DB][KVB];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int kb = 0; kb < KVB; ++kb) acc[i][kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Work items: (head of the group, query tile) pairs, query tiles from the
  // first one that can see row kvt * BKVD.
  const int ntq = (p.N + kTileRows - 1) / kTileRows;
  const int qt0 = p.causal ? (kvt * BKVD) / kTileRows : 0;
  const int per_head = ntq - qt0;
  const int items = R * per_head;
  const TileCopier<D> cp(wave, lane);
  const unsigned char* gQ = reinterpret_cast<const unsigned char*>(p.q);
  const unsigned char* gD = reinterpret_cast<const unsigned char*>(p.dout);
  const size_t qrow = (size_t)p.q_stride * 2, drow = (size_t)p.o_stride * 2;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)smem;
  // The log-sum-exp and Dd of an item's 64 query rows travel with its tiles:
  // wave 0 copies them (one word per lane, rows past the end clamped) into the
  // stage's row area, 256 bytes each, behind the four tiles of the two stages.
  const uint32_t rows0 = lds0 + 4 * TL::BYTES;
  auto issue = [&](int it) {
    const int h = g * R + it / per_head, qt = qt0 + it % per_head;
    const uint32_t st = lds0 + (it & 1) * 2 * TL::BYTES;
    cp.issue(gQ + (size_t)b * p.N * qrow, qrow, (uint32_t)(h * D * 2), qt * kTileRows, p.N, wave,
             lane, st);
    cp.issue(gD + (size_t)b * p.N * drow, drow, (uint32_t)(h * D * 2), qt * kTileRows, p.N, wave,
             lane, st + TL::BYTES);
    if (wave == 0) {
      const size_t row0 = ((size_t)b * p.H + h) * p.N;
      const uint32_t off = (uint32_t)min(qt * kTileRows + lane, p.N - 1) * 4;
      copy_dword_to_lds(p.lse + row0, off, rows0 + (it & 1) * 512);
      copy_dword_to_lds(p.Dd + row0, off, rows0 + (it & 1) * 512 + 256);
    }
  };
  const FragOffsets<D> fo(fr, grp);

  auto lds_at = [](int a) { return (const lds_u8*)(size_t)(uint32_t)a; };
  if (items > 0) issue(0);
  for (int it = 0; it < items; ++it) {
    KL_WAIT_VMCNT(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __syncthreads();
    if (it + 1 < items) issue(it + 1);
    const int qt = qt0 + it % per_head;
    const int q0 = qt * kTileRows;
    if (p.causal && q0 + kTileRows - 1 < kv0) continue;  // every row of the tile is before ours
    // Fragment offsets from this item's stage: one v_xad_u32 forms a read's
    // whole address (the dO tile and the row blocks are immediate offsets).
    const FragOffsets<D> fi = fo.at(lds0 + (it & 1) * 2 * TL::BYTES);
    const int rows_it = rows0 + (it & 1) * 512;
    const bool tail = q0 + kTileRows > p.N;
    // Tiles that reach this wave's value rows on the diagonal mask the weights
    // of later value rows (one uniform test per block of weights).
    const bool diag = p.causal && q0 < kv0 + 16 * KVB - 1;
    // Two 32-row query steps; each is one K = 32 step of the dV products.
#pragma unroll
    for (int qs = 0; qs < 2; ++qs) {
      bf16x8_t pp[KVB], ps[KVB];
      u32x4 wp[KVB], wsv[KVB];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int qb = 2 * qs + hh;  // 16-row query block of the tile
        f32x4_t sc[KVB], dp[KVB];
#pragma unroll
        for (int kb = 0; kb < KVB; ++kb) {
          sc[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
          dp[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        // Reads run two k-steps ahead of the products (fenced, order pinned).
        __builtin_amdgcn_sched_barrier(0);
        bf16x8_t aq[KS], ad[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const lds_u8* a = lds_at(fi.s(ks)) + qb * 16 * TL::ROW;
          aq[ks] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(a);
          ad[ks] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t*>(a + TL::BYTES);
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int kb = 0; kb < KVB; ++kb) {
            sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq[ks], vf[kb][ks], sc[kb], 0, 0, 0);
            dp[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad[ks], vf[kb][ks], dp[kb], 0, 0, 0);
          }
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
#pragma unroll
        for (int ks = 0; ks + 2 < KS; ++ks) {
          __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2 * KVB, 0);
          __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 4 * KVB, 0);
        __builtin_amdgcn_sched_barrier(0);
        // Lane: query rows q0 + 16 qb + 4 grp + r against value row kv0 + 16 kb + fr.
        // This block's rows 16 qb + 4 grp .. + 3: lse in log2 units (rows past the
        // sequence's end, copies of row N - 1 in the tile, get +inf, so their
        // weights and dS are exactly zero) and tau Dd.
        const f32x4_t lv = *reinterpret_cast<const __attribute__((address_space(3))) f32x4_t*>(
            lds_at(rows_it) + (qb * 16 + grp * 4) * 4);
        const f32x4_t dv4 = *reinterpret_cast<const __attribute__((address_space(3))) f32x4_t*>(
            lds_at(rows_it) + 256 + (qb * 16 + grp * 4) * 4);
        float l2[4], dq[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          l2[r] = lv[r] * kLog2e;
          if (tail) l2[r] = (q0 + qb * 16 + grp * 4 + r < p.N) ? l2[r] : INFINITY;
          dq[r] = dv4[r] * p.scale;
        }
        float pr[KVB][4];
#pragma unroll
        for (int kb = 0; kb < KVB; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) pr[kb][r] = fast_exp2(sc[kb][r] * c - l2[r]);
        if (diag) {
#pragma unroll
          for (int kb = 0; kb < KVB; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (kv0 + kb * 16 + fr > q0 + qb * 16 + grp * 4 + r) pr[kb][r] = 0.f;
        }
#pragma unroll
        for (int kb = 0; kb < KVB; ++kb) {
          float ds[4];
          // tau dS = P (tau dP - tau Dd)
#pragma unroll
          for (int r = 0; r < 4; ++r) ds[r] = pr[kb][r] * fmaf(dp[kb][r], p.scale, -dq[r]);
          wp[kb][2 * hh] = pack2(pr[kb][0], pr[kb][1]);
          wp[kb][2 * hh + 1] = pack2(pr[kb][2], pr[kb][3]);
          wsv[kb][2 * hh] = pack2(ds[0], ds[1]);
          wsv[kb][2 * hh + 1] = pack2(ds[2], ds[3]);
        }
      }
#pragma unroll
      for (int kb = 0; kb < KVB; ++kb) {
        pp[kb] = __builtin_bit_cast(bf16x8_t, wp[kb]);
        ps[kb] = __builtin_bit_cast(bf16x8_t, wsv[kb]);
      }
      // dV^T[d][kv] += dO^T P + Q~^T (tau dS) over query rows 32 qs + {4 grp .., 16 + 4 grp ..}.
      // Transposed reads run two column blocks ahead of the products.
      auto rd = [&](const int db, bf16x8_t& ad, bf16x8_t& aq) {
        const lds_u8* a = lds_at(fi.t(db)) + qs * 32 * TL::ROW;
        typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
        const s16x4 dlo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a + TL::BYTES));
        const s16x4 dhi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a + TL::BYTES + 16 * TL::ROW));
        const s16x4 qlo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)a);
        const s16x4 qhi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a + 16 * TL::ROW));
        ad = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(dlo, dhi, 0, 1, 2, 3, 4, 5, 6, 7));
        aq = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(qlo, qhi, 0, 1, 2, 3, 4, 5, 6, 7));
      };
      // The block is fenced (nothing moves across the fences) and its order
      // pinned: reads of blocks 0 and 1, then (products of db, reads of db + 2).
      __builtin_amdgcn_sched_barrier(0);
      bf16x8_t ad[DB], aq[DB];
      rd(0, ad[0], aq[0]);
      rd(1, ad[1], aq[1]);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        if (db + 2 < DB) rd(db + 2, ad[db + 2], aq[db + 2]);
#pragma unroll
        for (int kb = 0; kb < KVB; ++kb) {
          acc[db][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad[db], pp[kb], acc[db][kb], 0, 0, 0);
          acc[db][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq[db], ps[kb], acc[db][kb], 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 8, 0);
#pragma unroll
      for (int db = 0; db + 2 < DB; ++db) {
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2 * KVB, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
      }
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 4 * KVB, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // Lane holds dV^T[16 db + 4 grp + r][kv0 + 16 kb + fr].
  uint16_t* __restrict__ out = reinterpret_cast<uint16_t*>(p.dv);
#pragma unroll
  for (int kb = 0; kb < KVB; ++kb) {
    const int kv = kv0 + kb * 16 + fr;
    if (kv >= p.N) continue;
    uint16_t* dst = out + ((size_t)b * p.N + kv) * p.dv_stride + (size_t)g * D + grp * 4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const u32x2 w{pack2(acc[db][kb][0], acc[db][kb][1]), pack2(acc[db][kb][2], acc[db][kb][3])};
      *reinterpret_cast<u32x2*>(dst + db * 16) = w;
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 (and any dtype): VALU, one thread per query row (dQ~) or value row (dV)
// ---------------------------------------------------------------------------

template <typename T, int D>
__global__ __launch_bounds__(64) void bwd_dq_simple_kernel(BwdParams p) {
  const int i0 = blockIdx.x * 64;
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (p.H / p.G);
  const int i = i0 + threadIdx.x;
  const bool live = i < p.N;
  const T* Q = reinterpret_cast<const T*>(p.q);
  const T* V = reinterpret_cast<const T*>(p.v);
  const T* G = reinterpret_cast<const T*>(p.dout);
  __shared__ float sV[64][D];
  float q[D], go[D], acc[D];
  float l2 = 0.f, dd = 0.f;
  if (live) {
    l2 = p.lse[((size_t)b * p.H + h) * p.N + i] * kLog2e;
    dd = p.Dd[((size_t)b * p.H + h) * p.N + i];
  }
#pragma unroll
  for (int c = 0; c < D; ++c) {
    q[c] = live ? ldx(Q, ((size_t)b * p.N + i) * p.q_stride + (size_t)h * D + c) * p.scale_log2 : 0.f;
    go[c] = live ? ldx(G, ((size_t)b * p.N + i) * p.o_stride + (size_t)h * D + c) : 0.f;
    acc[c] = 0.f;
  }
  const int jend = p.causal ? min(p.N, i0 + 64) : p.N;
  for (int j0 = 0; j0 < jend; j0 += 64) {
    __syncthreads();
    for (int e = threadIdx.x; e < 64 * D; e += 64) {
      const int jj = e / D, c = e % D, j = j0 + jj;
      sV[jj][c] = j < p.N ? ldx(V, ((size_t)b * p.N + j) * p.v_stride + (size_t)g * D + c) : 0.f;
    }
    __syncthreads();
    const int jmax = min(64, (p.causal ? min(i + 1, p.N) : p.N) - j0);
    for (int jj = 0; jj < jmax; ++jj) {
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) {
        s = fmaf(q[c], sV[jj][c], s);
        dp = fmaf(go[c], sV[jj][c], dp);
      }
      const float ds = fast_exp2(s - l2) * (dp - dd);
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = fmaf(ds, sV[jj][c], acc[c]);
    }
  }
  if (live) {
    T* out = reinterpret_cast<T*>(p.dq);
#pragma unroll
    for (int c = 0; c < D; ++c)
      stx(out, ((size_t)b * p.N + i) * p.dq_stride + (size_t)h * D + c, acc[c] * p.scale);
  }
}

template <typename T, int D>
__global__ __launch_bounds__(64) void bwd_dv_simple_kernel(BwdParams p) {
  const int j0 = blockIdx.x * 64;
  const int g = blockIdx.y, b = blockIdx.z;
  const int R = p.H / p.G;
  const int j = j0 + threadIdx.x;
  const bool live = j < p.N;
  const T* Q = reinterpret_cast<const T*>(p.q);
  const T* V = reinterpret_cast<const T*>(p.v);
  const T* G = reinterpret_cast<const T*>(p.dout);
  __shared__ float sQ[32][D];
  __shared__ float sG[32][D];
  __shared__ float sL[32], sD[32];
  float v[D], acc[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    v[c] = live ? ldx(V, ((size_t)b * p.N + j) * p.v_stride + (size_t)g * D + c) : 0.f;
    acc[c] = 0.f;
  }
  const int ibeg = p.causal ? j0 : 0;
  for (int h = g * R; h < g * R + R; ++h) {
    for (int i0 = ibeg; i0 < p.N; i0 += 32) {
      __syncthreads();
      for (int e = threadIdx.x; e < 32 * D; e += 64) {
        const int ii = e / D, c = e % D, i = i0 + ii;
        const bool ok = i < p.N;
        sQ[ii][c] = ok ? ldx(Q, ((size_t)b * p.N + i) * p.q_stride + (size_t)h * D + c) : 0.f;
        sG[ii][c] = ok ? ldx(G, ((size_t)b * p.N + i) * p.o_stride + (size_t)h * D + c) : 0.f;
      }
      if (threadIdx.x < 32) {
        const int i = i0 + threadIdx.x;
        const bool ok = i < p.N;
        sL[threadIdx.x] = ok ? p.lse[((size_t)b * p.H + h) * p.N + i] * kLog2e : 0.f;
        sD[threadIdx.x] = ok ? p.Dd[((size_t)b * p.H + h) * p.N + i] : 0.f;
      }
      __syncthreads();
      const int imax = min(32, p.N - i0);
      for (int ii = 0; ii < imax; ++ii) {
        if (p.causal && i0 + ii < j) continue;
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) {
          s = fmaf(sQ[ii][c], v[c], s);
          dp = fmaf(sG[ii][c], v[c], dp);
        }
        const float pr = fast_exp2(s * p.scale_log2 - sL[ii]);
        const float ds = pr * (dp - sD[ii]) * p.scale;
#pragma unroll
        for (int c = 0; c < D; ++c) acc[c] = fmaf(pr, sG[ii][c], fmaf(ds, sQ[ii][c], acc[c]));
      }
    }
  }
  if (live) {
    T* out = reinterpret_cast<T*>(p.dv);
#pragma unroll
    for (int c = 0; c < D; ++c) stx(out, ((size_t)b * p.N + j) * p.dv_stride + (size_t)g * D + c, acc[c]);
  }
}

template <typename T, int D>
hipError_t launch_simple(const BwdParams& p, hipStream_t st) {
  hipLaunchKernelGGL((bwd_dq_simple_kernel<T, D>), dim3((p.N + 63) / 64, p.H, p.B), dim3(64), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((bwd_dv_simple_kernel<T, D>), dim3((p.N + 63) / 64, p.G, p.B), dim3(64), 0, st, p);
  return hipGetLastError();
}

template <int D>
hipError_t launch_mfma(const BwdParams& p, hipStream_t st) {
  using TL = AttnTile<D, kTileRows>;
  if (p.out_f32)
    hipLaunchKernelGGL((bwd_dq_kernel<D, false>), dim3(p.H, (p.N + BQD - 1) / BQD, p.B),
                       dim3(kThreads), NSTAGE * TL::BYTES, st, p);
  else
    hipLaunchKernelGGL((bwd_dq_kernel<D, true>), dim3(p.H, (p.N + BQD - 1) / BQD, p.B),
                       dim3(kThreads), NSTAGE * TL::BYTES, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  constexpr int dv_lds = 4 * TL::BYTES + 1024;  // two stages of Q~ and dO tiles, lse and Dd rows
  if (dv_lds > 65536) {
    static std::atomic<uint32_t> done{0};
    e = set_max_lds(reinterpret_cast<const void*>(bwd_dv_kernel<D>), dv_lds, done);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(bwd_dv_kernel<D>, dim3(p.G, (p.N + BKVD - 1) / BKVD, p.B), dim3(kThreads),
                     dv_lds, st, p);
  return hipGetLastError();
}

template <typename TO, typename T>
hipError_t launch_prep_t(const BwdParams& p, hipStream_t st) {
  const long rows = (long)p.B * p.N * p.H;
  const dim3 grid((unsigned)((rows + 15) / 16));
  if (p.D == 128) hipLaunchKernelGGL((bwd_prep_kernel<TO, T, 128>), grid, dim3(256), 0, st, p);
  else hipLaunchKernelGGL((bwd_prep_kernel<TO, T, 64>), grid, dim3(256), 0, st, p);
  return hipGetLastError();
}
template <typename T>
hipError_t launch_prep(const BwdParams& p, hipStream_t st) {
  return p.out_f32 ? launch_prep_t<float, T>(p, st) : launch_prep_t<T, T>(p, st);
}

}  // namespace

bool attn_bwd_mfma_supported(const BwdParams& p) {
  return p.dtype == KL_BF16 && (p.D == 64 || p.D == 128) && p.q_stride % 8 == 0 &&
         p.v_stride % 8 == 0 && p.o_stride % 8 == 0 && p.dq_stride % 4 == 0 &&
         p.dv_stride % 4 == 0 && (size_t)p.v_stride * 2 * 8 < (1u << 31) &&
         (size_t)p.q_stride * 2 * 8 < (1u << 31) && (size_t)p.o_stride * 2 * 8 < (1u << 31);
}

hipError_t launch_attention_backward(const BwdParams& p, hipStream_t st) {
  if (p.B == 0 || p.N == 0) return hipSuccess;
  if (p.D != 64 && p.D != 128) return hipErrorInvalidValue;
  // Dd: on the matrix cores from the fp32 output when there is one (in the dQ~
  // kernel's prologue, which publishes it for the dV kernel), else from P and
  // dP in the dQ~ kernel's first sweep; on the vector ALU from the output (the
  // prep kernel).
  const bool mfma = attn_bwd_mfma_supported(p);
  if (!mfma) {
    hipError_t e = p.dtype == KL_BF16 ? launch_prep<uint16_t>(p, st) : launch_prep<float>(p, st);
    if (e != hipSuccess) return e;
  }
  if (mfma) return p.D == 128 ? launch_mfma<128>(p, st) : launch_mfma<64>(p, st);
  if (p.dtype == KL_BF16)
    return p.D == 128 ? launch_simple<uint16_t, 128>(p, st) : launch_simple<uint16_t, 64>(p, st);
  return p.D == 128 ? launch_simple<float, 128>(p, st) : launch_simple<float, 64>(p, st);
}

}  // namespace kl
