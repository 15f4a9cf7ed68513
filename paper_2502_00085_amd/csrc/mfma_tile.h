// Vector types, the LDS tile layout and wait-count immediates shared by the two
// matrix-core attention kernels (the decode kernel and the tree prefill kernel), gfx950.
#pragma once

#include "td_internal.h"

namespace td {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Physical 16-byte chunk of logical chunk c of tile row r: rows are rotated by whole
// 64-byte blocks so that the transposed reads of four consecutive rows hit four
// different groups of 16 banks.
template <int CPR, int NBLK>
__device__ inline int phys_chunk(int r, int c) {
  return (c + 4 * (r % NBLK)) % CPR;
}

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14,
// expcnt in 6:4, lgkmcnt in 11:8)
constexpr int kWaitVmAll = 0 | (7 << 4) | (15 << 8);                // vmcnt(0)
// vmcnt(n), 0 <= n < 64: at most n vector memory operations of this wave outstanding
constexpr int wait_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkmAll = 15 | (3 << 14) | (7 << 4) | (0 << 8);  // lgkmcnt(0)

}  // namespace td
