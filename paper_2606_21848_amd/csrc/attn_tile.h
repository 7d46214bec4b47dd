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

// Two floats rounded to bf16 (nearest even) and packed low, high.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 b2;
  b2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

}  // namespace kl
