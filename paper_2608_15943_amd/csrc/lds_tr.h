// LDS tiles read along their rows with the gfx950 transpose read (ds_read_b64_tr_b16),
// shared by the backward attention kernels and the GEMM's transposed-operand paths.
#pragma once

#include "common.h"

namespace kvp {

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// Staged tiles use a sub-tiled LDS layout: an NR x NC bf16 tile is stored as NC / 32 blocks
// of 32 columns, each NR rows of 64 bytes; 16-byte chunk k (0..3) of row r of a block sits
// at position k ^ ((r >> 2) & 3).  A column-block or 16-row offset is then a constant byte
// offset (so every read below is one lane register plus an immediate), and 16 consecutive
// rows of one chunk column cover all 64 banks.
template <int NR>
__device__ __forceinline__ int sub_off(int r, int c) {
    return (c >> 5) * (NR * 64) + r * 64 + ((((c >> 3) & 3) ^ ((r >> 2) & 3)) << 4) + ((c & 7) << 1);
}

// One 1 KB direct load (16 bytes per lane) of rows 16 q .. 16 q + 15 of column block sb:
// lane i fetches the global chunk that belongs at position i % 4 of row 16 q + i / 4.
// Returns the chunk index (0..3) within the block; the caller supplies the global row.
__device__ __forceinline__ int sub_chunk(int lane) { return (lane & 3) ^ ((lane >> 4) & 3); }

// 8 consecutive columns c .. c + 7 (c % 8 == 0) of row r: one 16-byte read.
template <int NR>
__device__ __forceinline__ bf16x8 row8(const u32x4* tile, int r, int c) {
    return *(const bf16x8*)((const char*)tile + sub_off<NR>(r, c));
}

// Operand fragment taken along a tile's rows: lane (n = lane % 32, hi = lane / 32) receives
// tile[r0 + 8 hi + j][c0 + n], j = 0..7 (with PERM, column c0 + swap_b23(n)); r0 % 16 == 0
// and c0 % 32 == 0.  Two ds_read_b64_tr_b16: in each group of 16 lanes, lane 4 a + e
// receives element e of the 8 bytes addressed by lanes a, a + 4, a + 8, a + 12 of the group,
// so lane i of a group addresses row r0 + 8 hi + i / 4 (+ 4 for the second read) at the
// 4-column block that the result lanes with a = i % 4 need.
template <int NR, bool PERM>
__device__ __forceinline__ bf16x8 tr_frag(const u32x4* tile, int r0, int c0, int lane) {
    const int G = lane >> 4, src = lane & 15, a = src & 3;
    const int ap = PERM ? (((a & 1) << 1) | (a >> 1)) : a;
    const int col = 16 * (G & 1) + 4 * ap;            // < 32
    const int row = 8 * (G >> 1) + (src >> 2);         // < 16
    const char* base = (const char*)tile + (c0 >> 5) * (NR * 64) + r0 * 64;
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base + sub_off<NR>(row, col)));
    const v4i16 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base + sub_off<NR>(row + 4, col)));
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
}

}  // namespace kvp
