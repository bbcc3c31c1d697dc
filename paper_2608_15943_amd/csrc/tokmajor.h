// Token-major copies of a wave's [32 tokens][128 dims] bf16 output block, written through
// the wave's own 8 KB of LDS ([128 dims][32 tokens]) so that each dimension's 32 tokens
// leave as four 16-byte runs instead of 2-byte stores scattered over 128 rows.
// The attention kernels use it for O^T (forward) and [dQ|dK|dV]^T (backward), the operands
// of the weight-gradient products.  Call sites must have finished their own LDS reads of the
// region (a workgroup barrier) before the first put.
#pragma once

#include "common.h"

namespace kvp {

// Lane holding token `tok` (0..31): dims d0 .. d0 + 3 of it, packed as in the row-major store.
__device__ __forceinline__ void tm_put_token(uint16_t* ts, int d0, int tok, u32x2 w) {
    ts[(d0 + 0) * 32 + tok] = (uint16_t)(w[0] & 0xFFFFu);
    ts[(d0 + 1) * 32 + tok] = (uint16_t)(w[0] >> 16);
    ts[(d0 + 2) * 32 + tok] = (uint16_t)(w[1] & 0xFFFFu);
    ts[(d0 + 3) * 32 + tok] = (uint16_t)(w[1] >> 16);
}

// Lane holding dim `d`: tokens k4 .. k4 + 3 (k4 % 4 == 0) of it.
__device__ __forceinline__ void tm_put_dim(uint16_t* ts, int d, int k4, u32x2 w) {
    *(u32x2*)&ts[d * 32 + k4] = w;
}

// Row row0 + d of out (ld entries per row) receives the block's tokens t0 .. t0 + 31 of dim d,
// those below nvalid only; t0 and ld are multiples of 8.
__device__ __forceinline__ void tm_flush(const uint16_t* ts, uint16_t* out, size_t ld, int row0, size_t t0,
                                         int nvalid, int lane) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int idx = 64 * i + lane, d = idx >> 2, c = idx & 3;
        const u32x4 v = *(const u32x4*)&ts[d * 32 + 8 * c];
        uint16_t* dst = out + (size_t)(row0 + d) * ld + t0 + 8 * c;
        if (8 * c + 8 <= nvalid) {
            *(u32x4*)dst = v;
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (8 * c + j < nvalid) dst[j] = (uint16_t)((v[j >> 1] >> (16 * (j & 1))) & 0xFFFFu);
        }
    }
}

}  // namespace kvp
