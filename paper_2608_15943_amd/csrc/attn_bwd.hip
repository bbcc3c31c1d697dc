// Backward of the KV-shared attention layer on bf16 matrix cores (gfx950), d_h = 128.
//
// With S = Q K^T (masked), P = softmax(S / sqrt(d)) and O = P V (Sec. 2.2, Eq. 2), the
// gradients are dV = P^T dO, dP = dO V^T, dS = P * (dP - D) with D = rowsum(dO * O),
// dQ = dS K / sqrt(d) and dK = dS^T Q / sqrt(d).  P is rebuilt from the row
// log-sum-exp the forward kernel saved.  A layer's dK and dV belong to the layer that
// owns the K/V slot it read (Eq. 3): a consumer adds its share into an fp32 buffer of
// its producer, and the producer's own launch adds that buffer to its share and writes
// the result.  RoPE is orthogonal per position, so its transpose (a rotation by
// -pos * theta) is applied to dQ and dK in the epilogues, before any accumulation.
//
// Kernels:
//   attn_bwd_prep    D, and the transposed copies dO^T, Q^T, O^T the products over
//                    the query axis need (each [a*128][B*Sp], Sp = S rounded up to 64,
//                    zero past S).
//   flash_bwd_kv     one workgroup per (sequence, KV head, 256 keys); loops over the r
//                    query heads of the group and the query blocks at or after its
//                    keys; dK, dV accumulate in registers.
//   flash_bwd_q      one workgroup per (sequence, head, 256 queries); loops over the
//                    key blocks at or before its queries; dQ accumulates in registers.
//   transpose_bf16   batched, zero-padded 2-D transposes (activations, weights, caches).
//
// Operand layouts follow from v_mfma_f32_32x32x16_bf16: an operand lane holds 8
// consecutive elements of the reduction axis, and an accumulator lane holds one output
// column.  The first product of each kernel reads its A rows in a permuted order (bits 2
// and 3 of the row swapped), so that the 8 values a lane holds for each 16-wide step of
// the second product are 8 consecutive positions: P and dS feed the next products
// straight from registers, and the other operand is one 16-byte LDS read.
#include <math.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

constexpr int D = 128;

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

__device__ __forceinline__ int swap_b23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// 16 bytes per lane, global -> LDS; lane i lands at lds_base + 16 i.
__device__ __forceinline__ void load_lds16(const void* g, void* lds_base) {
    __builtin_amdgcn_global_load_lds((gvoid_t*)g, (lvoid_t*)lds_base, 16, 0, 0);
}
// 4 bytes per lane; lane i lands at lds_base + 4 i.
__device__ __forceinline__ void load_lds4(const void* g, void* lds_base) {
    __builtin_amdgcn_global_load_lds((gvoid_t*)g, (lvoid_t*)lds_base, 4, 0, 0);
}

// 8 fp32 -> bf16x8 (round to nearest even).
__device__ __forceinline__ bf16x8 pack8(const float* e) {
    u32x4 w;
    w[0] = pack2bf(e[0], e[1]);
    w[1] = pack2bf(e[2], e[3]);
    w[2] = pack2bf(e[4], e[5]);
    w[3] = pack2bf(e[6], e[7]);
    return as_bf16x8(w);
}

// ---------------------------------------------------------------------------
// Batched 2-D transpose: out[p][c][r] = in[p][r][c] for r < R, c < C, and 0 for
// R <= r < Rp or C <= c < Cp.  64 x 64 tiles through LDS.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ in,
                                                        uint16_t* __restrict__ out, int R, int C,
                                                        size_t in_ld, size_t in_plane, size_t out_ld,
                                                        size_t out_plane, int Rp, int Cp, int tiles_r) {
    __shared__ uint16_t t[64][66];
    const int p = blockIdx.z;
    const int r0 = (blockIdx.x % tiles_r) * 64, c0 = blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const uint16_t* src = in + (size_t)p * in_plane;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int r = r0 + ty + 4 * k, c = c0 + tx;
        t[ty + 4 * k][tx] = (r < R && c < C) ? src[(size_t)r * in_ld + c] : (uint16_t)0;
    }
    __syncthreads();
    uint16_t* dst = out + (size_t)p * out_plane;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int c = c0 + ty + 4 * k, r = r0 + tx;
        if (c < Cp && r < Rp) dst[(size_t)c * out_ld + r] = t[tx][ty + 4 * k];
    }
}

__global__ __launch_bounds__(256) void f32_to_bf16_kernel(const float* __restrict__ x,
                                                          uint16_t* __restrict__ y, size_t n) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
        y[i] = f2bf(x[i]);
}

// out[row-block b][m][n] = sum over the planes of part[s][m][n]; rows [0, rows0) go to
// dst0, the next rows1 to dst1, the rest to dst2 (each [rows_i][N], fp32).
__global__ __launch_bounds__(256) void reduce_planes_kernel(const float* __restrict__ part, int planes,
                                                            size_t plane, int M, int N, float* dst0,
                                                            int rows0, float* dst1, int rows1,
                                                            float* dst2) {
    const size_t n4 = (size_t)M * N / 4;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
        f32x4 s = *(const f32x4*)(part + 4 * i);
        for (int k = 1; k < planes; ++k) s += *(const f32x4*)(part + k * plane + 4 * i);
        const size_t e = 4 * i;
        const int m = (int)(e / N);
        const int n = (int)(e - (size_t)m * N);
        float* dst;
        int lm;
        if (m < rows0) { dst = dst0; lm = m; }
        else if (m < rows0 + rows1) { dst = dst1; lm = m - rows0; }
        else { dst = dst2; lm = m - rows0 - rows1; }
        *(f32x4*)(dst + (size_t)lm * N + n) = s;
    }
}

// ---------------------------------------------------------------------------
// D = rowsum(dO * O) and the transposed copies.  One workgroup per (sequence, head,
// 64 positions); the three [64][128] tiles pass through LDS.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void attn_bwd_prep_kernel(const uint16_t* __restrict__ dO,
                                                            const uint16_t* __restrict__ O,
                                                            const uint16_t* __restrict__ Q,
                                                            float* __restrict__ dsum,
                                                            uint16_t* __restrict__ dOt,
                                                            uint16_t* __restrict__ Qt,
                                                            uint16_t* __restrict__ Ot, int B, int S,
                                                            int Sp, int a) {
    __shared__ uint16_t tile[3][64][136];   // rows of 128 values + 8 of padding
    const int nst = Sp / 64;
    const int st = blockIdx.x % nst, bh = blockIdx.x / nst;
    const int b = bh / a, head = bh - b * a;
    const int s0 = st * 64;
    const int tid = threadIdx.x;
    const size_t ld = (size_t)a * D;
    // Loads: thread t reads 4 x 16 bytes of row t / 4 (dims 32 (t % 4) .. + 31) of each tile.
    const int r = tid >> 2, q4 = tid & 3;
    const int s = s0 + r;
    float acc = 0.f;
    if (s < S) {
        const size_t off = ((size_t)b * S + s) * ld + head * D + 32 * q4;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const u32x4 vd = *(const u32x4*)(dO + off + 8 * k);
            const u32x4 vo = *(const u32x4*)(O + off + 8 * k);
            const u32x4 vq = *(const u32x4*)(Q + off + 8 * k);
            *(u32x4*)&tile[0][r][32 * q4 + 8 * k] = vd;
            *(u32x4*)&tile[1][r][32 * q4 + 8 * k] = vq;
            *(u32x4*)&tile[2][r][32 * q4 + 8 * k] = vo;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc += __uint_as_float(vd[e] << 16) * __uint_as_float(vo[e] << 16);
                acc += __uint_as_float(vd[e] & 0xFFFF0000u) * __uint_as_float(vo[e] & 0xFFFF0000u);
            }
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int m = 0; m < 3; ++m) *(u32x4*)&tile[m][r][32 * q4 + 8 * k] = u32x4{0, 0, 0, 0};
    }
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    if (q4 == 0) dsum[((size_t)b * a + head) * Sp + s] = acc;
    __syncthreads();
    // Stores: output row d (of the head's 128), 8 positions per 16-byte store; thread t
    // writes rows t / 8 + 32 k, positions 8 (t % 8) .. + 7.
    const size_t ldt = (size_t)B * Sp;
    const int c8 = tid & 7;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int d = (tid >> 3) + 32 * k;
        const size_t off = (size_t)(head * D + d) * ldt + (size_t)b * Sp + s0 + 8 * c8;
#pragma unroll
        for (int m = 0; m < 3; ++m) {
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                w[e] = (uint32_t)tile[m][8 * c8 + 2 * e][d] | ((uint32_t)tile[m][8 * c8 + 2 * e + 1][d] << 16);
            uint16_t* dst = m == 0 ? dOt : (m == 1 ? Qt : Ot);
            *(u32x4*)(dst + off) = u32x4{w[0], w[1], w[2], w[3]};
        }
    }
}

// ---------------------------------------------------------------------------
// dK, dV.  Workgroup = 8 waves = 256 keys of one (sequence, KV head); wave w owns keys
// 32 w .. 32 w + 31 (one accumulator column each for dK and dV per lane: 4 blocks of
// 32 dims); two waves per SIMD.  The keys' V rows stay in LDS for the whole kernel
// ([256][128], 64 KB); K is held in registers.  Per step: one block of 32 queries of one
// of the r heads, staged in LDS as Q, dO ([32][128], 256-byte rows, chunk c at
// c ^ (row & 15)) and Q^T, dO^T ([128][32], 64-byte rows, chunk c at c ^ ((row >> 2) & 3)),
// plus the 32 log-sum-exp and D values; double buffered (2 x 32.25 KB).
//   S  [32 q x 32 k] = Q K^T     (A = Q rows, permuted; B = K, registers)
//   dP [32 q x 32 k] = dO V^T    (A = dO rows, same order; B = V rows, LDS)
//   dV [32 k x 128]  += P^T dO   (A = P from the S registers; B = dO^T, LDS)
//   dK [32 k x 128]  += dS^T Q   (A = dS; B = Q^T, LDS)
// ---------------------------------------------------------------------------
struct KvArgs {
    const uint16_t* q;      // [B*S][a*128] post-RoPE Q of the layer
    const uint16_t* qt;     // [a*128][B*Sp]
    const uint16_t* dO;     // [B*S][a*128]
    const uint16_t* dOt;    // [a*128][B*Sp]
    const float* lse;       // [B][a][Sp], log2 domain
    const float* dsum;      // [B][a][Sp]
    const uint16_t* kc;     // producer K slot [Bmax][g][cap][128]
    const uint16_t* vr;     // producer V rows [B*g][Sp][128], zero past S
    const float2* rope;     // [S][64]
    const float* acc_in_k;  // [B][g][S][128] or null
    const float* acc_in_v;
    float* acc_out_k;       // may alias acc_in_*
    float* acc_out_v;
    uint16_t* out;          // final rows [B*S][ldo] or null; dK at col_k + kvh*128, dV at col_v
    uint16_t* outT;         // final transposed [*][B*Sp] or null, same columns as rows
    int ldo, col_k, col_v;
    int B, S, Sp, a, g, cap;
    float scale_log2, scale;
};

constexpr int KV_BQ = 32, KV_BK = 256, KV_NT = 512;

__global__ __launch_bounds__(KV_NT, 2) void flash_bwd_kv_kernel(KvArgs A) {
    __shared__ u32x4 lvk[KV_BK * 16];          // V rows of the workgroup's keys
    __shared__ u32x4 lq[2][KV_BQ * 16];
    __shared__ u32x4 ldo_[2][KV_BQ * 16];
    __shared__ u32x4 lqt[2][D * 4];
    __shared__ u32x4 ldot[2][D * 4];
    __shared__ float lstat[2][2 * KV_BQ];      // [stage][lse 0..31, D 0..31]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;
    const int G = A.B * A.g;
    const int kb = blockIdx.x / G, grp = blockIdx.x - kb * G;   // heaviest key blocks first
    const int b = grp / A.g, kvh = grp - b * A.g;
    const int r = A.a / A.g;
    const int k0w = kb * KV_BK + 32 * wave;
    const int key = k0w + l32;                 // the key whose column this lane holds
    const bool kvalid = key < A.S;
    const size_t plane = (size_t)b * A.g + kvh;

    // V rows of the 256 keys into LDS (rows past Sp clamped: their keys are masked).
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int row = 32 * wave + 4 * j + (lane >> 4);
        const int c = (lane & 15) ^ (row & 15);
        const int pos = min(kb * KV_BK + row, A.Sp - 1);
        load_lds16(A.vr + (plane * A.Sp + pos) * D + 8 * c, &lvk[(32 * wave + 4 * j) * 16]);
    }
    // K of the lane's key as the B operand of S (8 dims per 16-wide step); zero past S.
    bf16x8 kf[8];
    {
        const uint16_t* krow = A.kc + (plane * A.cap + (kvalid ? key : 0)) * D + 8 * hi;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            u32x4 kw = *(const u32x4*)(krow + 16 * ks);
            if (!kvalid) kw = u32x4{0, 0, 0, 0};
            kf[ks] = as_bf16x8(kw);
        }
    }

    const int nqb = A.Sp / KV_BQ;
    const int qb_lo = min(kb * (KV_BK / KV_BQ), nqb);
    const int nq_h = nqb - qb_lo;               // query blocks per head
    const int n_it = r * nq_h;
    const size_t ld = (size_t)A.a * D, ldt = (size_t)A.B * A.Sp;

    auto issue = [&](int it, int stg) {
        const int head = kvh * r + it / nq_h;
        const int qb0 = (qb_lo + it % nq_h) * KV_BQ;
        {
            const int row = 4 * wave + (lane >> 4);
            const int c = (lane & 15) ^ (row & 15);
            const size_t src = ((size_t)b * A.S + min(qb0 + row, A.S - 1)) * ld + head * D + 8 * c;
            load_lds16(A.q + src, &lq[stg][(4 * wave) * 16]);
            load_lds16(A.dO + src, &ldo_[stg][(4 * wave) * 16]);
        }
        {
            const int d = 16 * wave + (lane >> 2);
            const int c = (lane & 3) ^ ((d >> 2) & 3);
            const size_t src = (size_t)(head * D + d) * ldt + (size_t)b * A.Sp + qb0 + 8 * c;
            load_lds16(A.qt + src, &lqt[stg][(16 * wave) * 4]);
            load_lds16(A.dOt + src, &ldot[stg][(16 * wave) * 4]);
        }
        if (wave == 0) {
            const float* src = (hi == 0 ? A.lse : A.dsum) + ((size_t)b * A.a + head) * A.Sp + qb0 + l32;
            load_lds4(src, &lstat[stg][0]);
        }
    };

    f32x16 dk[4], dv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        dk[i] = f32x16{};
        dv[i] = f32x16{};
    }
    const int rsw = swap_b23(l32);

    if (n_it > 0) issue(0, 0);
    for (int it = 0; it < n_it; ++it) {
        const int stg = it & 1;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();                          // tile it landed; tile it - 1 fully read
        if (it + 1 < n_it) issue(it + 1, stg ^ 1);
        const int qb0 = (qb_lo + it % nq_h) * KV_BQ;
        if (qb0 + KV_BQ - 1 < k0w) continue;      // every query of the block precedes the wave's keys
        f32x16 s = f32x16{}, dp = f32x16{};
        const int vr_ = 32 * wave + l32;          // this lane's key row in the V tile
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            const int c = (2 * ks + hi) ^ (rsw & 15);
            s = mfma32x32x16(as_bf16x8(lq[stg][rsw * 16 + c]), kf[ks], s);
            const bf16x8 vf = as_bf16x8(lvk[vr_ * 16 + ((2 * ks + hi) ^ (vr_ & 15))]);
            dp = mfma32x32x16(as_bf16x8(ldo_[stg][rsw * 16 + c]), vf, dp);
        }
        // Register i holds query qb0 + 16 (i / 8) + 8 hi + i % 8.
        bf16x8 pa[2], da[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int qo = 16 * h + 8 * hi;
            // Branch-free: the exponent is computed for every entry (masked ones may be
            // garbage) and the mask selects 0; the 8 statistics are two 16-byte reads each.
            const f32x4 l0 = *(const f32x4*)&lstat[stg][qo], l1 = *(const f32x4*)&lstat[stg][qo + 4];
            const f32x4 d0 = *(const f32x4*)&lstat[stg][KV_BQ + qo], d1 = *(const f32x4*)&lstat[stg][KV_BQ + qo + 4];
            float pe[8], de[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int qi = qb0 + qo + k;
                const float lse = k < 4 ? l0[k] : l1[k - 4], dd = k < 4 ? d0[k] : d1[k - 4];
                const bool vis = key <= qi && qi < A.S;
                const float e = __builtin_amdgcn_exp2f(fmaf(s[8 * h + k], A.scale_log2, -lse));
                pe[k] = vis ? e : 0.f;
                de[k] = vis ? e * (dp[8 * h + k] - dd) : 0.f;
            }
            pa[h] = pack8(pe);
            da[h] = pack8(de);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int d = 32 * nb + l32;
                const int ch = (2 * h + hi) ^ ((d >> 2) & 3);
                dv[nb] = mfma32x32x16(pa[h], as_bf16x8(ldot[stg][d * 4 + ch]), dv[nb]);
                dk[nb] = mfma32x32x16(da[h], as_bf16x8(lqt[stg][d * 4 + ch]), dk[nb]);
            }
    }

    // Epilogue: lane column d = 32 nb + l32; register e of block nb holds key
    // k0w + 8 (e / 4) + 4 hi + e % 4.  Scale, rotate dK back (pairs nb, nb + 2), add the
    // consumers' shares, write.
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int kk = k0w + 8 * (e >> 2) + 4 * hi + (e & 3);
        float yk[4], yv[4];
        if (kk < A.S) {
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                const float2 cs = A.rope[(size_t)kk * 64 + 32 * nb + l32];
                const float x1 = dk[nb][e] * A.scale, x2 = dk[nb + 2][e] * A.scale;
                yk[nb] = x1 * cs.x + x2 * cs.y;
                yk[nb + 2] = x2 * cs.x - x1 * cs.y;
            }
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) yv[nb] = dv[nb][e];
            const size_t ai = (((size_t)b * A.g + kvh) * A.S + kk) * D + l32;
            if (A.acc_in_k) {
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) {
                    yk[nb] += A.acc_in_k[ai + 32 * nb];
                    yv[nb] += A.acc_in_v[ai + 32 * nb];
                }
            }
            if (A.acc_out_k) {
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) {
                    A.acc_out_k[ai + 32 * nb] = yk[nb];
                    A.acc_out_v[ai + 32 * nb] = yv[nb];
                }
            }
            if (A.out) {
                uint16_t* row = A.out + ((size_t)b * A.S + kk) * A.ldo + kvh * D + l32;
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) {
                    row[A.col_k + 32 * nb] = f2bf(yk[nb]);
                    row[A.col_v + 32 * nb] = f2bf(yv[nb]);
                }
            }
        } else {
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) yk[nb] = yv[nb] = 0.f;
        }
        if (A.outT && kk < A.Sp) {
            const size_t col = (size_t)b * A.Sp + kk;
            const size_t ldt2 = (size_t)A.B * A.Sp;
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                A.outT[(size_t)(A.col_k + kvh * D + 32 * nb + l32) * ldt2 + col] = f2bf(yk[nb]);
                A.outT[(size_t)(A.col_v + kvh * D + 32 * nb + l32) * ldt2 + col] = f2bf(yv[nb]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// dQ.  Workgroup = 8 waves = 256 queries of one (sequence, head); wave w owns queries
// 32 w .. 32 w + 31 (lane: one query column).  Key blocks of 64 stream through LDS as
// K and V rows ([64][128], 256-byte rows) and K^T ([128][64], 128-byte rows), double
// buffered (2 x 48 KB).
//   S^T  [32 k x 32 q] x 2 = K Q^T      (A = K rows, permuted; B = Q, registers)
//   dP^T [32 k x 32 q] x 2 = V dO^T     (A = V rows, same order; B = dO, registers)
//   dQ^T [128 x 32 q]     += K^T dS^T   (A = K^T from LDS; B = dS^T from the registers)
// ---------------------------------------------------------------------------
struct QArgs {
    const uint16_t* q;      // [B*S][a*128]
    const uint16_t* dO;     // [B*S][a*128]
    const float* lse;       // [B][a][Sp]
    const float* dsum;      // [B][a][Sp]
    const uint16_t* kc;     // producer K slot [Bmax][g][cap][128]
    const uint16_t* kt;     // K^T [B*g][128][Sp], zero past S
    const uint16_t* vr;     // V rows [B*g][Sp][128], zero past S
    const float2* rope;     // [S][64]
    uint16_t* out;          // dQ rows [B*S][ldo] at column head*128, or null
    uint16_t* outT;         // dQ^T [a*128][B*Sp] (rows head*128 + d), or null
    int ldo;
    int B, S, Sp, a, g, cap;
    float scale_log2, scale;
};

constexpr int Q_BQ = 256, Q_BKV = 64, Q_NT = 512;

__global__ __launch_bounds__(Q_NT, 2) void flash_bwd_q_kernel(QArgs A) {
    __shared__ u32x4 lk[2][Q_BKV * 16];
    __shared__ u32x4 lv[2][Q_BKV * 16];
    __shared__ u32x4 lkt[2][D * 8];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;
    const int nqt = (A.S + Q_BQ - 1) / Q_BQ;
    const int BA = A.B * A.a;
    const int qt = nqt - 1 - blockIdx.x / BA;           // heaviest query tiles first
    const int rest = blockIdx.x - (blockIdx.x / BA) * BA;
    const int b = rest / A.a, head = rest - b * A.a;
    const int kvh = head / (A.a / A.g);
    const int q0w = qt * Q_BQ + 32 * wave;
    const int ql = q0w + l32;                           // the query of this lane's column
    const size_t ld = (size_t)A.a * D;

    bf16x8 qf[8], df[8];
    {
        const size_t row = ((size_t)b * A.S + min(ql, A.S - 1)) * ld + head * D + 8 * hi;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            qf[ks] = as_bf16x8(*(const u32x4*)(A.q + row + 16 * ks));
            df[ks] = as_bf16x8(*(const u32x4*)(A.dO + row + 16 * ks));
        }
    }
    const size_t si = ((size_t)b * A.a + head) * A.Sp + min(ql, A.Sp - 1);
    const float lse = A.lse[si], dd = A.dsum[si];

    const size_t plane = (size_t)b * A.g + kvh;
    const uint16_t* kbase = A.kc + plane * A.cap * D;
    const uint16_t* vbase = A.vr + plane * A.Sp * D;
    const uint16_t* tbase = A.kt + plane * D * A.Sp;
    const int last_q = min(qt * Q_BQ + Q_BQ - 1, A.S - 1);
    const int ntiles = last_q / Q_BKV + 1;

    auto issue = [&](int t, int stg) {
        const int t0 = t * Q_BKV;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int row = 8 * wave + 4 * j + (lane >> 4);
            const int c = (lane & 15) ^ (row & 15);
            load_lds16(kbase + (size_t)(t0 + row) * D + 8 * c, &lk[stg][(8 * wave + 4 * j) * 16]);
            load_lds16(vbase + (size_t)(t0 + row) * D + 8 * c, &lv[stg][(8 * wave + 4 * j) * 16]);
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int d = 16 * wave + 8 * j + (lane >> 3);
            const int c = (lane & 7) ^ ((d >> 1) & 7);
            load_lds16(tbase + (size_t)d * A.Sp + t0 + 8 * c, &lkt[stg][(16 * wave + 8 * j) * 8]);
        }
    };

    f32x16 dq[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) dq[i] = f32x16{};
    const int rsw = swap_b23(l32);

    issue(0, 0);
    for (int t = 0; t < ntiles; ++t) {
        const int stg = t & 1;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (t + 1 < ntiles) issue(t + 1, stg ^ 1);
        const int t0 = t * Q_BKV;
        if (t0 > q0w + 31 || q0w >= A.S) continue;    // no key of the block is visible to the wave
        f32x16 s[2], dp[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            s[mb] = f32x16{};
            dp[mb] = f32x16{};
            const int row = 32 * mb + rsw;
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const int c = (2 * ks + hi) ^ (row & 15);
                s[mb] = mfma32x32x16(as_bf16x8(lk[stg][row * 16 + c]), qf[ks], s[mb]);
                dp[mb] = mfma32x32x16(as_bf16x8(lv[stg][row * 16 + c]), df[ks], dp[mb]);
            }
        }
        // Register i of block mb holds key t0 + 32 mb + 16 (i / 8) + 8 hi + i % 8.
        bf16x8 db_[4];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                float de[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int kk = t0 + 32 * mb + 16 * h + 8 * hi + k;
                    const bool vis = kk <= ql && ql < A.S;
                    const float e = __builtin_amdgcn_exp2f(fmaf(s[mb][8 * h + k], A.scale_log2, -lse));
                    de[k] = vis ? e * (dp[mb][8 * h + k] - dd) : 0.f;
                }
                db_[2 * mb + h] = pack8(de);
            }
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int d = 32 * m + l32;
                const int ch = (2 * c + hi) ^ ((d >> 1) & 7);
                dq[m] = mfma32x32x16(as_bf16x8(lkt[stg][d * 8 + ch]), db_[c], dq[m]);
            }
    }

    // Epilogue: lane column = query ql; register e of block m holds dim
    // 32 m + 8 (e / 4) + 4 hi + e % 4.  Scale, rotate back (pairs m, m + 2), write.
    if (ql < A.Sp) {
        const bool valid = ql < A.S;
        const size_t col = (size_t)b * A.Sp + ql, ldt = (size_t)A.B * A.Sp;
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            float y[4][4];   // [block m][e % 4]
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int e4 = 0; e4 < 4; ++e4) {
                    const int e = 4 * g4 + e4;
                    const int i = 32 * m + 8 * g4 + 4 * hi + e4;
                    const float2 cs = valid ? A.rope[(size_t)ql * 64 + i] : float2{1.f, 0.f};
                    const float x1 = dq[m][e] * A.scale, x2 = dq[m + 2][e] * A.scale;
                    y[m][e4] = valid ? x1 * cs.x + x2 * cs.y : 0.f;
                    y[m + 2][e4] = valid ? x2 * cs.x - x1 * cs.y : 0.f;
                }
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int d0 = 32 * m + 8 * g4 + 4 * hi;
                if (A.out && valid) {
                    u32x2 w;
                    w[0] = pack2bf(y[m][0], y[m][1]);
                    w[1] = pack2bf(y[m][2], y[m][3]);
                    *(u32x2*)(A.out + ((size_t)b * A.S + ql) * A.ldo + head * D + d0) = w;
                }
                if (A.outT) {
#pragma unroll
                    for (int e4 = 0; e4 < 4; ++e4)
                        A.outT[(size_t)(head * D + d0 + e4) * ldt + col] = f2bf(y[m][e4]);
                }
            }
        }
    }
}

}  // namespace

hipError_t transpose_bf16(const uint16_t* in, uint16_t* out, int planes, int R, int C, size_t in_ld,
                          size_t in_plane, size_t out_ld, size_t out_plane, int Rp, int Cp,
                          hipStream_t st) {
    const int tr = (Rp + 63) / 64, tc = (Cp + 63) / 64;
    if (planes < 1 || tr < 1 || tc < 1) return hipSuccess;
    hipLaunchKernelGGL(transpose_kernel, dim3(tr, tc, planes), dim3(256), 0, st, in, out, R, C, in_ld,
                       in_plane, out_ld, out_plane, Rp, Cp, tr);
    return hipGetLastError();
}

hipError_t f32_to_bf16(const float* x, uint16_t* y, size_t n, hipStream_t st) {
    const int grid = (int)std::min<size_t>((n + 255) / 256, 4096);
    if (grid < 1) return hipSuccess;
    hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(grid), dim3(256), 0, st, x, y, n);
    return hipGetLastError();
}

hipError_t reduce_planes(const float* part, int planes, int M, int N, float* dst0, int rows0, float* dst1,
                         int rows1, float* dst2, hipStream_t st) {
    const size_t n4 = (size_t)M * N / 4;
    const int grid = (int)std::min<size_t>((n4 + 255) / 256, 8192);
    if (grid < 1) return hipSuccess;
    hipLaunchKernelGGL(reduce_planes_kernel, dim3(grid), dim3(256), 0, st, part, planes, (size_t)M * N, M,
                       N, dst0, rows0, dst1, rows1, dst2);
    return hipGetLastError();
}

hipError_t attn_bwd_prep_bf16(const uint16_t* dO, const uint16_t* O, const uint16_t* Q, float* dsum,
                              uint16_t* dOt, uint16_t* Qt, uint16_t* Ot, int B, int S, int Sp, int a,
                              hipStream_t st) {
    hipLaunchKernelGGL(attn_bwd_prep_kernel, dim3(B * a * (Sp / 64)), dim3(256), 0, st, dO, O, Q, dsum,
                       dOt, Qt, Ot, B, S, Sp, a);
    return hipGetLastError();
}

hipError_t flash_bwd_kv_bf16(const AttnBwdKv& p, hipStream_t st) {
    KvArgs A;
    A.q = p.q; A.qt = p.qt; A.dO = p.dO; A.dOt = p.dOt; A.lse = p.lse; A.dsum = p.dsum;
    A.kc = p.kc; A.vr = p.vr; A.rope = p.rope;
    A.acc_in_k = p.acc_in_k; A.acc_in_v = p.acc_in_v; A.acc_out_k = p.acc_out_k; A.acc_out_v = p.acc_out_v;
    A.out = p.out; A.outT = p.outT; A.ldo = p.ldo; A.col_k = p.col_k; A.col_v = p.col_v;
    A.B = p.B; A.S = p.S; A.Sp = p.Sp; A.a = p.a; A.g = p.g; A.cap = p.cap;
    A.scale = (float)(1.0 / sqrt((double)D));
    A.scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    const int nkb = (p.S + KV_BK - 1) / KV_BK;
    hipLaunchKernelGGL(flash_bwd_kv_kernel, dim3(nkb * p.B * p.g), dim3(KV_NT), 0, st, A);
    return hipGetLastError();
}

hipError_t flash_bwd_q_bf16(const AttnBwdQ& p, hipStream_t st) {
    QArgs A;
    A.q = p.q; A.dO = p.dO; A.lse = p.lse; A.dsum = p.dsum; A.kc = p.kc; A.kt = p.kt; A.vr = p.vr;
    A.rope = p.rope; A.out = p.out; A.outT = p.outT; A.ldo = p.ldo;
    A.B = p.B; A.S = p.S; A.Sp = p.Sp; A.a = p.a; A.g = p.g; A.cap = p.cap;
    A.scale = (float)(1.0 / sqrt((double)D));
    A.scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    const int nqt = (p.S + Q_BQ - 1) / Q_BQ;
    hipLaunchKernelGGL(flash_bwd_q_kernel, dim3(nqt * p.B * p.a), dim3(Q_NT), 0, st, A);
    return hipGetLastError();
}

}  // namespace kvp
