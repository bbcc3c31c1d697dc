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
//   attn_bwd_prep    D = rowsum(dO * O) per (token, head).
//   transpose_bf16   weight transposes for the dO and dX products.
//   flash_bwd_kv     one workgroup per (sequence, KV head, 256 keys); loops over the r
//                    query heads of the group and the query blocks at or after its
//                    keys; dK, dV accumulate in registers.
//   flash_bwd_q      one workgroup per (sequence, head, 256 queries); loops over the
//                    key blocks at or before its queries; dQ accumulates in registers.
//
// Operand layouts follow from v_mfma_f32_32x32x16_bf16: an operand lane holds 8
// consecutive elements of the reduction axis, and an accumulator lane holds one output
// column.  The first product of each kernel reads its A rows in a permuted order (bits 2
// and 3 of the row swapped), so that the 8 values a lane holds for each 16-wide step of
// the second product are 8 consecutive positions: P and dS feed the next products
// straight from registers.  Operands that run along a staged tile's rows (dO, Q and V^T
// for dV, dK and dP; K and V^T in the dQ kernel) are read with the LDS transpose read of
// gfx950, so every tile is staged once, in the layout it has in memory.
//
// Inside the loops the LDS fragment reads are placed by hand ahead of the products that
// consume them (the compiled order waited for every fragment right before its MFMA), and
// the causal mask is applied only in the blocks that touch the diagonal or the end of the
// sequence, behind a wave-uniform branch; every other block computes P and dS unmasked.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "lds_tr.h"
#include "tokmajor.h"

namespace kvp {
namespace {

constexpr int D = 128;

// LDS reads placed by hand (the dK, dV and the dQ kernels): a transposed read moves 8 bytes
// per lane, a row read 16, each from a per-lane address plus an immediate offset; a wait
// names the fragments it completes as in/out operands, so the MFMA that reads one cannot be
// scheduled before it.  LDS reads return in order, so a wait for at most N outstanding
// operations completes every read but the last N issued.
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
template <int OFF>
__device__ __forceinline__ u32x2_t tr_read(uint32_t addr) {
    u32x2_t v;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
    return v;
}
template <int N>
__device__ __forceinline__ void lgkm_wait2(u32x2_t& lo, u32x2_t& up) {
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(lo), "+v"(up) : "i"(N));
}
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<N, I + 1>(f);
    }
}
template <int OFF>
__device__ __forceinline__ u32x4 ds_read16(uint32_t addr) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
    return v;
}
template <int N>
__device__ __forceinline__ void lgkm_wait4(u32x4& a, u32x4& b, u32x2_t& c, u32x2_t& d) {
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) : "i"(N));
}
template <int N>
__device__ __forceinline__ void lgkm_wait3(u32x4& a, u32x2_t& b, u32x2_t& c) {
    asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(a), "+v"(b), "+v"(c) : "i"(N));
}
__device__ __forceinline__ bf16x8 join_frag(u32x2_t lo, u32x2_t up) {
    return __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], up[0], up[1]});
}

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

// out[c][r] = in[r][c]: 64 x 64 tiles through LDS (weights, once per layer).
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ in,
                                                        uint16_t* __restrict__ out, int R, int C,
                                                        size_t in_ld, size_t out_ld) {
    __shared__ uint16_t t[64][66];
    const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int r = r0 + ty + 4 * k, c = c0 + tx;
        t[ty + 4 * k][tx] = (r < R && c < C) ? in[(size_t)r * in_ld + c] : (uint16_t)0;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int c = c0 + ty + 4 * k, r = r0 + tx;
        if (c < C && r < R) out[(size_t)c * out_ld + r] = t[tx][ty + 4 * k];
    }
}

// The same for R, C multiples of 64 and 16-byte aligned rows: 16-byte global accesses (a
// lane reads 8 elements of a row and writes 8 of a transposed row).
__global__ __launch_bounds__(256) void transpose16_kernel(const uint16_t* __restrict__ in,
                                                          uint16_t* __restrict__ out, size_t in_ld,
                                                          size_t out_ld) {
    __shared__ uint16_t t[64][65];
    const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
    const int tid = threadIdx.x, seg = tid & 7, row = tid >> 3;   // 8 lanes per 64-element row
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int r = row + 32 * k;
        const u32x4 v = *(const u32x4*)(in + (size_t)(r0 + r) * in_ld + c0 + 8 * seg);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            t[r][8 * seg + 2 * e] = (uint16_t)(v[e] & 0xFFFFu);
            t[r][8 * seg + 2 * e + 1] = (uint16_t)(v[e] >> 16);
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int c = row + 32 * k;   // output row c0 + c holds input column c0 + c
        u32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = (uint32_t)t[8 * seg + 2 * e][c] | ((uint32_t)t[8 * seg + 2 * e + 1][c] << 16);
        *(u32x4*)(out + (size_t)(c0 + c) * out_ld + r0 + 8 * seg) = v;
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
// D = rowsum(dO * O) for every (token, head): each group of 16 lanes takes one pair, 8
// dims per lane (16 bytes of dO and of O), summed across the group.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void attn_bwd_prep_kernel(const uint16_t* __restrict__ dO,
                                                            const uint16_t* __restrict__ O,
                                                            float* __restrict__ dsum, int B, int S,
                                                            int Sp, int a) {
    const int M = B * S;
    const size_t ld = (size_t)a * D;
    const int item = blockIdx.x * 16 + (threadIdx.x >> 4);      // (token, head) pair
    const int sub = threadIdx.x & 15;
    const int m = item / a, head = item - (item / a) * a;
    float acc = 0.f;
    if (m < M) {
        const size_t off = (size_t)m * ld + head * D + 8 * sub;
        const u32x4 vd = *(const u32x4*)(dO + off);
        const u32x4 vo = *(const u32x4*)(O + off);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc += __uint_as_float(vd[e] << 16) * __uint_as_float(vo[e] << 16);
            acc += __uint_as_float(vd[e] & 0xFFFF0000u) * __uint_as_float(vo[e] & 0xFFFF0000u);
        }
    }
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
    if (sub == 0 && m < M) {
        const int b = m / S, s = m - b * S;
        dsum[((size_t)b * a + head) * Sp + s] = acc;
    }
}

// ---------------------------------------------------------------------------
// dK, dV.  Workgroup = 8 waves = 256 keys of one (sequence, KV head); wave w owns keys
// 32 w .. 32 w + 31 (one accumulator column each for dK and dV per lane: 4 blocks of
// 32 dims); two waves per SIMD.  K of the lane's key is held in registers, V^T of the 256
// keys in LDS ([128][256], 64 KB) for the whole kernel.  Per step: one block of 64
// queries of one of the r heads, staged in LDS as Q and dO rows ([64][128]) plus their 64
// log-sum-exp and D values; double buffered (2 x 32.5 KB); tiles in the sub-tiled layout.
// Each 32-query half:
//   S  [32 q x 32 k] = Q K^T     (A = Q rows, permuted; B = K, registers)
//   dP [32 q x 32 k] = dO V^T    (A = dO rows, same order; B = V^T tile along its rows)
//   dV [32 k x 128]  += P^T dO   (A = P from the S registers; B = dO tile along its rows)
//   dK [32 k x 128]  += dS^T Q   (A = dS; B = Q tile along its rows)
// The operands taken along a tile's rows are transposed reads (tr_frag), so no transposed
// copy of Q, dO or V is made.
// ---------------------------------------------------------------------------
struct KvArgs {
    const uint16_t* q;      // [B*S][a*128] post-RoPE Q of the layer
    const uint16_t* dO;     // [B*S][a*128]
    const float* lse;       // [B][a][Sp], log2 domain
    const float* dsum;      // [B][a][Sp]
    const uint16_t* kc;     // producer K slot [Bmax][g][cap][128]
    const uint16_t* vc;     // producer V slot [Bmax][g][128][cap]
    const float2* rope;     // [S][64]
    const float* acc_in_k;  // [B][g][S][128] or null
    const float* acc_in_v;
    float* acc_out_k;       // may alias acc_in_*
    float* acc_out_v;
    uint16_t* out;          // final rows [B*S][ldo] or null; dK at col_k + kvh*128, dV at col_v
    uint16_t* out_t;        // null, or the same values token-major [ldo][B*S] (S % 8 == 0)
    int ldo, col_k, col_v;
    int B, S, Sp, a, g, cap;
    float scale_log2, scale;
};

constexpr int KV_BQ = 64, KV_BK = 256, KV_NT = 512;

__global__ __launch_bounds__(KV_NT, 2) void flash_bwd_kv_kernel(KvArgs A) {
    __shared__ u32x4 lvt[D * 32];              // V^T of the workgroup's keys, 512-byte rows
    __shared__ u32x4 lq[2][KV_BQ * 16];
    __shared__ u32x4 ldo_[2][KV_BQ * 16];
    __shared__ float lstat[2][2 * KV_BQ];      // [stage][lse 0..63, D 0..63]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;
    const int G = A.B * A.g;
    const int kb = blockIdx.x / G, grp = blockIdx.x - kb * G;   // heaviest key blocks first
    const int b = grp / A.g, kvh = grp - b * A.g;
    const int r = A.a / A.g;
    const int k0w = kb * KV_BK + 32 * wave;
    const int k0u = __builtin_amdgcn_readfirstlane(k0w);   // the same value, held as wave-uniform
    const int key = k0w + l32;                 // the key whose column this lane holds
    const bool kvalid = key < A.S;
    const size_t plane = (size_t)b * A.g + kvh;

    // V^T of the 256 keys into LDS: wave w fills column block w (its own keys).  Chunks
    // past the slot are clamped: their keys lie beyond S, so their dP columns are masked.
    const int ch = sub_chunk(lane);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int row = 16 * q + (lane >> 2);
        const int k0 = min(kb * KV_BK + 32 * wave + 8 * ch, A.cap - 8);
        load_lds16(A.vc + (plane * D + row) * A.cap + k0, (char*)lvt + wave * (D * 64) + q * 1024);
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
    const size_t ld = (size_t)A.a * D;

    auto issue = [&](int it, int stg) {
        const int head = kvh * r + it / nq_h;
        const int qb0 = (qb_lo + it % nq_h) * KV_BQ;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int t = 2 * wave + j, sb = t >> 2, q = t & 3;
            const int row = 16 * q + (lane >> 2);
            const size_t src = ((size_t)b * A.S + min(qb0 + row, A.S - 1)) * ld + head * D + 32 * sb + 8 * ch;
            load_lds16(A.q + src, (char*)lq[stg] + sb * (KV_BQ * 64) + q * 1024);
            load_lds16(A.dO + src, (char*)ldo_[stg] + sb * (KV_BQ * 64) + q * 1024);
        }
        if (wave < 2) {
            const float* src = (wave == 0 ? A.lse : A.dsum) + ((size_t)b * A.a + head) * A.Sp + qb0 + lane;
            load_lds4(src, &lstat[stg][KV_BQ * wave]);
        }
    };

    f32x16 dk[4], dv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        dk[i] = f32x16{};
        dv[i] = f32x16{};
    }
    const int rsw = swap_b23(l32);
    // The transposed-read lane offsets of tr_frag<KV_BQ, false> (row r0 = 0, column block 0):
    // the rest of a fragment's address is an immediate.
    const int tr_row = 8 * (lane >> 5) + ((lane & 15) >> 2), tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int tr_lo = sub_off<KV_BQ>(tr_row, tr_col), tr_up = sub_off<KV_BQ>(tr_row + 4, tr_col);
    // Row chunks of row8<KV_BQ>(tile, rsw, 16 ks + 8 hi) for even and odd ks (block 0, rows
    // 0..31), and the V^T fragment of tr_frag<D, false>(lvt, 16 ks, 32 wave) at ks = 0.
    const int rc0 = sub_off<KV_BQ>(rsw, 8 * hi), rc1 = sub_off<KV_BQ>(rsw, 16 + 8 * hi);
    const uint32_t av_lo = (uint32_t)(uintptr_t)((const char*)lvt + wave * (D * 64) + sub_off<D>(tr_row, tr_col)),
                   av_up = (uint32_t)(uintptr_t)((const char*)lvt + wave * (D * 64) + sub_off<D>(tr_row + 4, tr_col));

    if (n_it > 0) issue(0, 0);
    // Per-lane LDS addresses in stage 0 (stage 1 is a constant offset further: the loop below
    // takes the stage as a compile-time constant): the two transposed reads of a dO / Q
    // fragment (row block 0, column block 0), and the lane's Q / dO row chunk (row rsw,
    // chunk 2 (ks & 1) + hi).  The k step's block, the half's rows and the stage are immediates.
    const uint32_t o_lo = (uint32_t)(uintptr_t)((const char*)ldo_[0] + tr_lo),
                   o_up = (uint32_t)(uintptr_t)((const char*)ldo_[0] + tr_up),
                   q_lo = (uint32_t)(uintptr_t)((const char*)lq[0] + tr_lo),
                   q_up = (uint32_t)(uintptr_t)((const char*)lq[0] + tr_up);
    const uint32_t aq0 = (uint32_t)(uintptr_t)((const char*)lq[0] + rc0),
                   aq1 = (uint32_t)(uintptr_t)((const char*)lq[0] + rc1),
                   ao0 = (uint32_t)(uintptr_t)((const char*)ldo_[0] + rc0),
                   ao1 = (uint32_t)(uintptr_t)((const char*)ldo_[0] + rc1);
    constexpr int kStage = KV_BQ * 16 * 16;   // bytes of one stage of lq / ldo_
    auto iteration = [&](int it, auto stg_t) __attribute__((always_inline)) {
        constexpr int stg = decltype(stg_t)::value;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();                          // tile it landed; tile it - 1 fully read
        if (it + 1 < n_it) issue(it + 1, stg ^ 1);
        const int qb0 = (qb_lo + it % nq_h) * KV_BQ;
        auto half = [&](auto rb_t) __attribute__((always_inline)) {
            constexpr int RB = decltype(rb_t)::value;
            const int rb = RB;
            if (qb0 + 32 * rb + 31 < k0w) return;   // every query of the half precedes the wave's keys
            // Wave-uniform: some entry of the half is masked (a query before one of the wave's
            // keys, or past S).  Most halves lie wholly below the diagonal and skip the mask.
            const int q_first = qb0 + 32 * rb;
            const bool masked = !(q_first >= k0u + 31 && q_first + 31 < A.S);
            f32x16 s = f32x16{}, dp = f32x16{};
            // S = Q K^T and dP = dO V^T over 8 k steps; step ks reads a Q row chunk, a dO row
            // chunk and a V^T fragment (two transposed reads), one step ahead of its products.
            {
                u32x4 fq[2], fo[2];
                u32x2_t fvl[2], fvu[2];
                auto rd = [&](auto ks_t) __attribute__((always_inline)) {
                    constexpr int ks = decltype(ks_t)::value;
                    constexpr int roff = stg * kStage + (ks >> 1) * (KV_BQ * 64) + 2048 * RB, voff = ks * 1024;
                    fq[ks % 2] = ds_read16<roff>(ks & 1 ? aq1 : aq0);
                    fo[ks % 2] = ds_read16<roff>(ks & 1 ? ao1 : ao0);
                    fvl[ks % 2] = tr_read<voff>(av_lo);
                    fvu[ks % 2] = tr_read<voff>(av_up);
                };
                rd(std::integral_constant<int, 0>{});
                static_for<8>([&](auto ks_t) __attribute__((always_inline)) {
                    constexpr int ks = decltype(ks_t)::value;
                    if constexpr (ks + 1 < 8) {
                        rd(std::integral_constant<int, ks + 1>{});
                        lgkm_wait4<4>(fq[ks % 2], fo[ks % 2], fvl[ks % 2], fvu[ks % 2]);
                    } else {
                        lgkm_wait4<0>(fq[ks % 2], fo[ks % 2], fvl[ks % 2], fvu[ks % 2]);
                    }
                    s = mfma32x32x16(as_bf16x8(fq[ks % 2]), kf[ks], s);
                    dp = mfma32x32x16(as_bf16x8(fo[ks % 2]), join_frag(fvl[ks % 2], fvu[ks % 2]), dp);
                });
            }
            // Register i holds query qb0 + 32 rb + 16 (i / 8) + 8 hi + i % 8.
            bf16x8 pa[2], da[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int qo = 32 * rb + 16 * h + 8 * hi;
                // Branch-free: the exponent is computed for every entry (masked ones may be
                // garbage) and the mask selects 0; the 8 statistics are two 16-byte reads each.
                const f32x4 l0 = *(const f32x4*)&lstat[stg][qo], l1 = *(const f32x4*)&lstat[stg][qo + 4];
                const f32x4 d0 = *(const f32x4*)&lstat[stg][KV_BQ + qo];
                const f32x4 d1 = *(const f32x4*)&lstat[stg][KV_BQ + qo + 4];
                float pe[8], de[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const float lse = k < 4 ? l0[k] : l1[k - 4], dd = k < 4 ? d0[k] : d1[k - 4];
                    const float e = __builtin_amdgcn_exp2f(fmaf(s[8 * h + k], A.scale_log2, -lse));
                    pe[k] = e;
                    de[k] = e * (dp[8 * h + k] - dd);
                }
                if (masked) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int qi = qb0 + qo + k;
                        const bool vis = key <= qi && qi < A.S;
                        pe[k] = vis ? pe[k] : 0.f;
                        de[k] = vis ? de[k] : 0.f;
                    }
                }
                pa[h] = pack8(pe);
                da[h] = pack8(de);
            }
            // dV += P^T dO, dK += dS^T Q: 16 products, product i = (h, nb, dV or dK) =
            // (i / 8, i / 2 % 4, i % 2), each B fragment two transposed reads.  The reads go two
            // products ahead through three rotating fragments (the compiled order waited for
            // each fragment right before its product).
            {
                u32x2_t flo[3], fup[3];
                auto issue = [&](auto i_t) __attribute__((always_inline)) {
                    constexpr int i = decltype(i_t)::value;
                    constexpr int h = i / 8, nb = (i / 2) % 4;
                    constexpr int off = stg * kStage + nb * (KV_BQ * 64) + (32 * RB + 16 * h) * 64;
                    const uint32_t a_lo = (i % 2) ? q_lo : o_lo, a_up = (i % 2) ? q_up : o_up;
                    flo[i % 3] = tr_read<off>(a_lo);
                    fup[i % 3] = tr_read<off>(a_up);
                };
                issue(std::integral_constant<int, 0>{});
                issue(std::integral_constant<int, 1>{});
                static_for<16>([&](auto i_t) __attribute__((always_inline)) {
                    constexpr int i = decltype(i_t)::value;
                    constexpr int h = i / 8, nb = (i / 2) % 4;
                    if constexpr (i + 1 < 16) lgkm_wait2<2>(flo[i % 3], fup[i % 3]);
                    else lgkm_wait2<0>(flo[i % 3], fup[i % 3]);
                    if constexpr (i + 2 < 16) issue(std::integral_constant<int, i + 2>{});
                    const bf16x8 f = join_frag(flo[i % 3], fup[i % 3]);
                    if constexpr (i % 2 == 0) dv[nb] = mfma32x32x16(pa[h], f, dv[nb]);
                    else dk[nb] = mfma32x32x16(da[h], f, dk[nb]);
                });
            }
        };
        half(std::integral_constant<int, 0>{});
        half(std::integral_constant<int, 1>{});
    };
    for (int it = 0; it < n_it; it += 2) {
        iteration(it, std::integral_constant<int, 0>{});
        if (it + 1 < n_it) iteration(it + 1, std::integral_constant<int, 1>{});
    }

    // Epilogue: lane column d = 32 nb + l32; register e of block nb holds key
    // k0w + 8 (e / 4) + 4 hi + e % 4.  Scale, rotate dK back (pairs nb, nb + 2), add the
    // consumers' shares, write.
    // The token-major copy is staged per wave, dK in the V^T buffer and dV in the Q / dO
    // stages (all free once every wave is past its last block): the lane's 4 consecutive
    // keys of each dimension as one 8-byte LDS write.
    uint32_t tk[4][2], tv[4][2];             // the group's 4 keys, packed in pairs
    uint16_t* tsk = (uint16_t*)&lvt[0] + wave * (D * 32);
    uint16_t* tsv = wave < 4 ? (uint16_t*)&lq[0][0] + wave * (D * 32) : (uint16_t*)&ldo_[0][0] + (wave - 4) * (D * 32);
    if (A.out_t) __syncthreads();
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
                    const uint16_t bk = f2bf(yk[nb]), bv = f2bf(yv[nb]);
                    row[A.col_k + 32 * nb] = bk;
                    row[A.col_v + 32 * nb] = bv;
                    const int sh = 16 * (e & 1), ix = (e >> 1) & 1;
                    tk[nb][ix] = (e & 1) ? (tk[nb][ix] | ((uint32_t)bk << sh)) : (uint32_t)bk;
                    tv[nb][ix] = (e & 1) ? (tv[nb][ix] | ((uint32_t)bv << sh)) : (uint32_t)bv;
                }
            }
        }
        if ((e & 3) == 3 && A.out_t) {
            const int k4 = 8 * (e >> 2) + 4 * hi;    // the group's first key within the wave's 32
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                tm_put_dim(tsk, 32 * nb + l32, k4, u32x2{tk[nb][0], tk[nb][1]});
                tm_put_dim(tsv, 32 * nb + l32, k4, u32x2{tv[nb][0], tv[nb][1]});
            }
        }
    }
    if (A.out_t) {
        const size_t ldt = (size_t)A.B * A.S, t0 = (size_t)b * A.S + k0w;
        tm_flush(tsk, A.out_t, ldt, A.col_k + kvh * D, t0, A.S - k0w, lane);
        tm_flush(tsv, A.out_t, ldt, A.col_v + kvh * D, t0, A.S - k0w, lane);
    }
}

// ---------------------------------------------------------------------------
// dQ.  Workgroup = 8 waves = 256 queries of one (sequence, head); wave w owns queries
// 32 w .. 32 w + 31 (lane: one query column).  Key blocks of 128 stream through LDS as
// K rows and V^T rows straight from the producer's slot ([128][128] each, sub-tiled
// layout), double buffered (2 x 64 KB).  Each 64-key half:
//   S^T  [32 k x 32 q] x 2 = K Q^T      (A = K rows, permuted; B = Q, registers)
//   dP^T [32 k x 32 q] x 2 = V dO^T     (A = V^T tile along its rows, same order; B = dO)
//   dQ^T [128 x 32 q]     += K^T dS^T   (A = K tile along its rows; B = dS^T, registers)
// ---------------------------------------------------------------------------
struct QArgs {
    const uint16_t* q;      // [B*S][a*128]
    const uint16_t* dO;     // [B*S][a*128]
    const float* lse;       // [B][a][Sp]
    const float* dsum;      // [B][a][Sp]
    const uint16_t* kc;     // producer K slot [Bmax][g][cap][128]
    const uint16_t* vc;     // producer V slot [Bmax][g][128][cap]
    const float2* rope;     // [S][64]
    uint16_t* out;          // dQ rows [B*S][ldo] at column head*128
    uint16_t* out_t;        // null, or dQ token-major [ldo][B*S] (S % 8 == 0)
    int ldo;
    int B, S, Sp, a, g, cap;
    float scale_log2, scale;
};

constexpr int Q_BQ = 256, Q_BKV = 128, Q_NT = 512;

__global__ __launch_bounds__(Q_NT, 2) void flash_bwd_q_kernel(QArgs A) {
    __shared__ u32x4 lk[2][Q_BKV * 16];
    __shared__ u32x4 lvt[2][D * 16];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;
    const int nqt = (A.S + Q_BQ - 1) / Q_BQ;
    const int BA = A.B * A.a;
    const int qt = nqt - 1 - blockIdx.x / BA;           // heaviest query tiles first
    const int rest = blockIdx.x - (blockIdx.x / BA) * BA;
    const int b = rest / A.a, head = rest - b * A.a;
    const int kvh = head / (A.a / A.g);
    const int q0w = qt * Q_BQ + 32 * wave;
    const int q0u = __builtin_amdgcn_readfirstlane(q0w);   // the same value, held as wave-uniform
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
    const uint16_t* vbase = A.vc + plane * D * A.cap;
    const int last_q = min(qt * Q_BQ + Q_BQ - 1, A.S - 1);
    const int ntiles = last_q / Q_BKV + 1;

    // K rows past S are replaced by row S - 1 (finite: they meet dS = 0 in dQ); V^T chunks
    // past the slot are clamped (their keys' dP rows are masked).
    const int ch = sub_chunk(lane);
    auto issue = [&](int t, int stg) {
        const int t0 = t * Q_BKV;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int u = 4 * wave + j, sb = u >> 3, q = u & 7;
            const int row = 16 * q + (lane >> 2);
            load_lds16(kbase + (size_t)min(t0 + row, A.S - 1) * D + 32 * sb + 8 * ch,
                       (char*)lk[stg] + sb * (Q_BKV * 64) + q * 1024);
            load_lds16(vbase + (size_t)row * A.cap + min(t0 + 32 * sb + 8 * ch, A.cap - 8),
                       (char*)lvt[stg] + sb * (D * 64) + q * 1024);
        }
    };

    f32x16 dq[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) dq[i] = f32x16{};
    const int rsw = swap_b23(l32);

    // Per-lane LDS addresses in stage 0 (stage 1 is a constant offset further: the loop below
    // takes the stage as a compile-time constant).  K row chunk of row8<Q_BKV>(lk, rsw,
    // 16 ks + 8 hi) for even and odd ks; the two transposed reads of tr_frag<D, true>(lvt, 0, 0)
    // and of tr_frag<Q_BKV, false>(lk, 0, 0).  Row blocks, column blocks, k steps and the
    // stage are immediates.
    const int G = lane >> 4, a4 = lane & 3;
    const int tr_row = 8 * (G >> 1) + ((lane & 15) >> 2);
    const int tr_col = 16 * (G & 1) + 4 * a4, trp_col = 16 * (G & 1) + 4 * (((a4 & 1) << 1) | (a4 >> 1));
    const uint32_t k_base = (uint32_t)(uintptr_t)lk[0], v_base = (uint32_t)(uintptr_t)lvt[0];
    const uint32_t ak0 = k_base + sub_off<Q_BKV>(rsw, 8 * hi), ak1 = k_base + sub_off<Q_BKV>(rsw, 16 + 8 * hi);
    const uint32_t pv_lo = v_base + sub_off<D>(tr_row, trp_col), pv_up = v_base + sub_off<D>(tr_row + 4, trp_col);
    const uint32_t tk_lo = k_base + sub_off<Q_BKV>(tr_row, tr_col), tk_up = k_base + sub_off<Q_BKV>(tr_row + 4, tr_col);
    constexpr int kStage = Q_BKV * 16 * 16;   // bytes of one stage of lk (and of lvt: D == Q_BKV)
    static_assert(D == Q_BKV, "one stage size for lk and lvt");

    auto tile = [&](int t, auto stg_t) __attribute__((always_inline)) {
        constexpr int stg = decltype(stg_t)::value;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (t + 1 < ntiles) issue(t + 1, stg ^ 1);
        const int t0 = t * Q_BKV;
        if (q0w >= A.S) return;
        auto half = [&](auto hf_t) __attribute__((always_inline)) {
            constexpr int HF = decltype(hf_t)::value;
            constexpr int k0 = 64 * HF;                     // first key of the half in the tile
            if (t0 + k0 > q0w + 31) return;                // no key of the half is visible
            // Wave-uniform: some entry of the half is masked (a key after one of the wave's
            // queries, or a query past S).  Halves wholly below the diagonal skip the mask.
            const bool masked = !(t0 + k0 + 63 <= q0u && q0u + 31 < A.S);
            f32x16 s[2], dp[2];
            // S = K Q^T and dP = V dO^T: 16 products, step j = (mb, ks) = (j / 8, j % 8) reads a
            // K row chunk and a V^T fragment (two transposed reads), one step ahead.
            {
                u32x4 fk[2];
                u32x2_t fvl[2], fvu[2];
                auto rd = [&](auto j_t) __attribute__((always_inline)) {
                    constexpr int j = decltype(j_t)::value, mb = j / 8, ks = j % 8;
                    constexpr int koff = stg * kStage + (ks >> 1) * (Q_BKV * 64) + (k0 + 32 * mb) * 64;
                    constexpr int voff = stg * kStage + ((k0 + 32 * mb) >> 5) * (D * 64) + ks * 1024;
                    fk[j % 2] = ds_read16<koff>(ks & 1 ? ak1 : ak0);
                    fvl[j % 2] = tr_read<voff>(pv_lo);
                    fvu[j % 2] = tr_read<voff>(pv_up);
                };
                s[0] = s[1] = dp[0] = dp[1] = f32x16{};
                rd(std::integral_constant<int, 0>{});
                static_for<16>([&](auto j_t) __attribute__((always_inline)) {
                    constexpr int j = decltype(j_t)::value, mb = j / 8, ks = j % 8;
                    if constexpr (j + 1 < 16) {
                        rd(std::integral_constant<int, j + 1>{});
                        lgkm_wait3<3>(fk[j % 2], fvl[j % 2], fvu[j % 2]);
                    } else {
                        lgkm_wait3<0>(fk[j % 2], fvl[j % 2], fvu[j % 2]);
                    }
                    s[mb] = mfma32x32x16(as_bf16x8(fk[j % 2]), qf[ks], s[mb]);
                    dp[mb] = mfma32x32x16(join_frag(fvl[j % 2], fvu[j % 2]), df[ks], dp[mb]);
                });
            }
            // Register i of block mb holds key t0 + k0 + 32 mb + 16 (i / 8) + 8 hi + i % 8.
            bf16x8 db_[4];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    float de[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const float e = __builtin_amdgcn_exp2f(fmaf(s[mb][8 * h + k], A.scale_log2, -lse));
                        de[k] = e * (dp[mb][8 * h + k] - dd);
                    }
                    if (masked) {
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            const int kk = t0 + k0 + 32 * mb + 16 * h + 8 * hi + k;
                            de[k] = kk <= ql && ql < A.S ? de[k] : 0.f;
                        }
                    }
                    db_[2 * mb + h] = pack8(de);
                }
            // dQ += dS K: 16 products, product i = (c, m) = (i / 4, i % 4), each K^T fragment two
            // transposed reads, two products ahead through three rotating fragments.
            {
                u32x2_t flo[3], fup[3];
                auto issue_k = [&](auto i_t) __attribute__((always_inline)) {
                    constexpr int i = decltype(i_t)::value, c = i / 4, m = i % 4;
                    constexpr int off = stg * kStage + m * (Q_BKV * 64) + (k0 + 16 * c) * 64;
                    flo[i % 3] = tr_read<off>(tk_lo);
                    fup[i % 3] = tr_read<off>(tk_up);
                };
                issue_k(std::integral_constant<int, 0>{});
                issue_k(std::integral_constant<int, 1>{});
                static_for<16>([&](auto i_t) __attribute__((always_inline)) {
                    constexpr int i = decltype(i_t)::value, c = i / 4, m = i % 4;
                    if constexpr (i + 1 < 16) lgkm_wait2<2>(flo[i % 3], fup[i % 3]);
                    else lgkm_wait2<0>(flo[i % 3], fup[i % 3]);
                    if constexpr (i + 2 < 16) issue_k(std::integral_constant<int, i + 2>{});
                    dq[m] = mfma32x32x16(join_frag(flo[i % 3], fup[i % 3]), db_[c], dq[m]);
                });
            }
        };
        half(std::integral_constant<int, 0>{});
        half(std::integral_constant<int, 1>{});
    };

    issue(0, 0);
    for (int t = 0; t < ntiles; t += 2) {
        tile(t, std::integral_constant<int, 0>{});
        if (t + 1 < ntiles) tile(t + 1, std::integral_constant<int, 1>{});
    }

    // Epilogue: lane column = query ql; register e of block m holds dim
    // 32 m + 8 (e / 4) + 4 hi + e % 4.  Scale, rotate back (pairs m, m + 2), write.  The
    // token-major copy is staged per wave in the K buffers (free once every wave is past
    // its last tile).
    uint16_t* ts = (uint16_t*)&lk[0][0] + wave * (D * 32);
    if (A.out_t) __syncthreads();
    if (ql < A.S) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            float y[4][4];   // [block m][e % 4]
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int e4 = 0; e4 < 4; ++e4) {
                    const int e = 4 * g4 + e4;
                    const int i = 32 * m + 8 * g4 + 4 * hi + e4;
                    const float2 cs = A.rope[(size_t)ql * 64 + i];
                    const float x1 = dq[m][e] * A.scale, x2 = dq[m + 2][e] * A.scale;
                    y[m][e4] = x1 * cs.x + x2 * cs.y;
                    y[m + 2][e4] = x2 * cs.x - x1 * cs.y;
                }
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int d0 = 32 * m + 8 * g4 + 4 * hi;
                u32x2 w;
                w[0] = pack2bf(y[m][0], y[m][1]);
                w[1] = pack2bf(y[m][2], y[m][3]);
                *(u32x2*)(A.out + ((size_t)b * A.S + ql) * A.ldo + head * D + d0) = w;
                if (A.out_t) tm_put_token(ts, d0, l32, w);
            }
        }
    }
    if (A.out_t)
        tm_flush(ts, A.out_t, (size_t)A.B * A.S, head * D, (size_t)b * A.S + q0w, A.S - q0w, lane);
}

}  // namespace

hipError_t transpose_bf16(const uint16_t* in, uint16_t* out, int R, int C, size_t in_ld, size_t out_ld,
                          hipStream_t st) {
    if (R < 1 || C < 1) return hipSuccess;
    const bool wide = R % 64 == 0 && C % 64 == 0 && in_ld % 8 == 0 && out_ld % 8 == 0 &&
                      ((reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out)) & 15) == 0;
    if (wide)
        hipLaunchKernelGGL(transpose16_kernel, dim3(R / 64, C / 64), dim3(256), 0, st, in, out, in_ld, out_ld);
    else
        hipLaunchKernelGGL(transpose_kernel, dim3((R + 63) / 64, (C + 63) / 64), dim3(256), 0, st, in, out, R, C,
                           in_ld, out_ld);
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

hipError_t attn_bwd_prep_bf16(const uint16_t* dO, const uint16_t* O, float* dsum, int B, int S, int Sp, int a,
                              hipStream_t st) {
    const int items = B * S * a;
    hipLaunchKernelGGL(attn_bwd_prep_kernel, dim3((items + 15) / 16), dim3(256), 0, st, dO, O, dsum, B, S, Sp, a);
    return hipGetLastError();
}

hipError_t flash_bwd_kv_bf16(const AttnBwdKv& p, hipStream_t st) {
    KvArgs A;
    A.q = p.q; A.dO = p.dO; A.lse = p.lse; A.dsum = p.dsum; A.kc = p.kc; A.vc = p.vc; A.rope = p.rope;
    A.acc_in_k = p.acc_in_k; A.acc_in_v = p.acc_in_v; A.acc_out_k = p.acc_out_k; A.acc_out_v = p.acc_out_v;
    A.out = p.out; A.out_t = p.out_t; A.ldo = p.ldo; A.col_k = p.col_k; A.col_v = p.col_v;
    if (p.out_t && (!p.out || p.S % 8 != 0)) return hipErrorInvalidValue;
    A.B = p.B; A.S = p.S; A.Sp = p.Sp; A.a = p.a; A.g = p.g; A.cap = p.cap;
    A.scale = (float)(1.0 / sqrt((double)D));
    A.scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    const int nkb = (p.S + KV_BK - 1) / KV_BK;
    hipLaunchKernelGGL(flash_bwd_kv_kernel, dim3(nkb * p.B * p.g), dim3(KV_NT), 0, st, A);
    return hipGetLastError();
}

hipError_t flash_bwd_q_bf16(const AttnBwdQ& p, hipStream_t st) {
    QArgs A;
    A.q = p.q; A.dO = p.dO; A.lse = p.lse; A.dsum = p.dsum; A.kc = p.kc; A.vc = p.vc;
    A.rope = p.rope; A.out = p.out; A.out_t = p.out_t; A.ldo = p.ldo;
    if (p.out_t && p.S % 8 != 0) return hipErrorInvalidValue;
    A.B = p.B; A.S = p.S; A.Sp = p.Sp; A.a = p.a; A.g = p.g; A.cap = p.cap;
    A.scale = (float)(1.0 / sqrt((double)D));
    A.scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    const int nqt = (p.S + Q_BQ - 1) / Q_BQ;
    hipLaunchKernelGGL(flash_bwd_q_kernel, dim3(nqt * p.B * p.a), dim3(Q_NT), 0, st, A);
    return hipGetLastError();
}

}  // namespace kvp
