// LDS tile layout shared by the attention kernels: ROWS rows of D bf16 values
// (D * 2 bytes each), moved from memory by direct-to-LDS copies of 1 KiB per
// wave instruction, with each row's 16-byte chunks XOR-swizzled so that both
// the row-fragment reads (16 rows, one chunk: ds_read_b128) and the
// transposing reads (ds_read_b64_tr_b16 over 4-row x 16-column blocks) hit
// distinct banks.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace kl {

template <int D, int ROWS>
struct AttnTile {
  static constexpr int ROW = D * 2;                // bytes per row
  static constexpr int CHUNKS = D / 8;             // 16-byte chunks per row
  static constexpr int BYTES = ROWS * ROW;         // one tile
  static constexpr int COPIES = BYTES / 1024 / 4;  // copy instructions per wave per tile (4 waves)
  // Physical chunk of logical chunk c in row r (depends on r mod 16 only).
  static __device__ __forceinline__ int swz(int r, int c) {
    if constexpr (D == 128) return c ^ (((r & 7) << 1) | ((r >> 3) & 1));
    else return c ^ ((r >> 1) & 7);
  }
  static __device__ __forceinline__ int off(int r, int c) { return r * ROW + (swz(r, c) << 4); }
};

// Per-lane LDS offsets of the two fragment reads, formed at each use from two
// registers instead of a table (a kernel near its register limit would keep a
// table in scratch). The row-fragment read (ds_read_b128) of lane (fr, grp) at
// k-step ks reads logical chunk 4 ks + grp of row fr + 16 kb; the transposing
// read (ds_read_b64_tr_b16) for column block db reads row 4 grp + fr / 4,
// columns 16 db + 4 (fr % 4). With the XOR swizzle of AttnTile:
//   off(r, 4 ks + grp)      = r ROW + 16 (grp ^ (key & 3)) + 64 (ks ^ (key >> 2))
//   off(r, 2 db + e) + 8 f  = r ROW + 16 (e ^ (key & 1)) + 8 f + 32 (db ^ (key >> 1))
// where key = swz(r, 0) is the row's swizzle key, e = (fr % 4) / 2, f = fr % 2.
template <int D>
struct FragOffsets {
  int sbase, skey;  // row-fragment reads: sbase + (64 ks ^ skey)
  int tbase, tkey;  // transposed reads:   tbase + (32 db ^ tkey)
  __device__ __forceinline__ FragOffsets(int fr, int grp) {
    using T = AttnTile<D, 16>;
    const int ks_key = T::swz(fr, 0);
    sbase = fr * T::ROW + 16 * (grp ^ (ks_key & 3));
    skey = (ks_key >> 2) << 6;
    const int r = grp * 4 + (fr >> 2);
    const int t_key = T::swz(r, 0);
    tbase = r * T::ROW + 16 * (((fr & 3) >> 1) ^ (t_key & 1)) + 8 * (fr & 1);
    tkey = (t_key >> 1) << 5;
  }
  // Volatile, so the compiler forms the offset at its use rather than hoisting
  // every variant out of the loop into registers.
  static __device__ __forceinline__ int xad(int key, int imm, int base) {
    int r;
    asm volatile("v_xad_u32 %0, %1, %2, %3" : "=v"(r) : "v"(key), "s"(imm), "v"(base));
    return r;
  }
  __device__ __forceinline__ int s(int ks) const { return xad(skey, ks << 6, sbase); }
  __device__ __forceinline__ int t(int db) const { return xad(tkey, db << 5, tbase); }
  // The same offsets relative to `base` (a tile's LDS address), so that a read
  // needs only the one v_xad_u32 for its whole address.
  __device__ __forceinline__ FragOffsets at(uint32_t base) const {
    FragOffsets f = *this;
    f.sbase += (int)base;
    f.tbase += (int)base;
    return f;
  }
};

// Two floats rounded to bf16 (nearest even) and packed low, high.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 b2;
  b2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

}  // namespace kl
