// Projection GEMMs of the prefill path on bf16 matrix cores (gfx950).
//
// C[M][N] = A[M][K] * W[N][K]^T with both operands K-contiguous ([out, in]
// weights), fp32 accumulation in v_mfma_f32_32x32x16_bf16, and two fused
// epilogues:
//   * QKV: Q of every layer and K, V of producers (Sec. 2.2, Eq. 1); RoPE is
//     applied to Q and K in registers (the rotate-half partner of column c
//     sits in the same lane, 64 columns on), then Q goes to its buffer, K to
//     the producer's cache slot and V, transposed, to the V slot.  A consumer
//     runs the same kernel with N = a * d_h (Q only).
//   * residual: X_{l+1} = X_l + O W_O^T, with the residual stream read and
//     written in fp32 between layers and a bf16 copy for the next projection.
//
// Tiling: 256 x 256 x 64 per workgroup of 4 waves (2 x 2, 128 x 128 each, a
// 4 x 4 grid of 32 x 32 MFMA blocks = 256 fp32 accumulators per lane).
// Operand tiles go straight from global memory into LDS (global_load_lds_dwordx4,
// no staging registers), double buffered (2 x 64 KB), one barrier per K step;
// LDS rows are 128 B with the 16-byte chunk index XOR-swizzled by
// ((row >> 1) & 7), which spreads the 32-row fragment reads over all 64 banks.  Tiles are ordered so that each XCD works on a contiguous group of
// M-panels (its own L2 keeps the A and W panels hot).
#include "common.h"
#include "kernels.h"
#include "lds_tr.h"

namespace kvp {
namespace {

constexpr int BM = 256, BN = 256, BK = 64, NT = 256, GROUP_M = 8;

// Word 3 of a raw buffer resource: a valid (32-bit) data format.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ const uint16_t* w_row(const WRows& w, int n, int K) {
    if (n < w.rows[0]) return (const uint16_t*)w.p[0] + (size_t)n * K;
    n -= w.rows[0];
    if (n < w.rows[1]) return (const uint16_t*)w.p[1] + (size_t)n * K;
    n -= w.rows[1];
    return (const uint16_t*)w.p[2] + (size_t)n * K;
}

// ---------------------------------------------------------------------------
// Epilogues.  After the main loop each wave owns a 128 x 128 fp32 tile in
// registers (lane: column n = 32 nb + l32, rows m = 32 mb + 8 (i/4) + 4 hi + i%4).
// stage() writes it into the wave's 32 KB of the (now idle) LDS and flush()
// copies it out with 16-byte coalesced global accesses, in Epi::kPasses passes.
// ---------------------------------------------------------------------------

// fp32 staging rows (128 x 64 fp32 = 256-byte rows, 16-byte chunk c): lanes write 128
// contiguous bytes of rows m and m + 4, and read one chunk of 4 rows per 16 lanes; this
// XOR keeps both patterns free of bank conflicts on the 64-bank LDS.
__device__ __forceinline__ int f32_pos(int m, int c) {
    return c ^ ((m & 1) | ((((m >> 1) ^ (m >> 2)) & 1) << 3));
}
__device__ __forceinline__ void st_f32(char* st, int m, int n, float v) {
    *(float*)(st + m * 256 + f32_pos(m, n >> 2) * 16 + (n & 3) * 4) = v;
}
__device__ __forceinline__ u32x4 ld_f32(const char* st, int m, int c) {
    return *(const u32x4*)(st + m * 256 + f32_pos(m, c) * 16);
}

// Q, K (rotated) and V (transposed) of the projection GEMM.  Q/K tiles go through LDS as
// fp32 in two passes; pass h holds head columns 32 h .. 32 h + 31 and their rotate-half
// partners 64 + 32 h .. 64 + 32 h + 31, so RoPE is applied in the flush with the cos/sin
// of each (position, column) read as contiguous table rows.  V is staged once, in bf16,
// transposed ([n][m], 8-byte unit u of row n at position u ^ (n & 31)).
struct QkvEpi {
    static constexpr int kPasses = 2;
    // cos/sin rows of the lane's 8 Q/K items, requested before the tile is staged.
    struct Pre {
        u32x4 cs[8][4];
    };
    QkvOut o;
    __device__ __forceinline__ void set_split(int) {}
    // Element offsets of K row s and of V^T element (dimension n, position s) of
    // sequence b, KV head `head`: in the contiguous slot or in s's page.
    __device__ __forceinline__ size_t k_row(int b, int head, int s) const {
        if (o.pages.pt)
            return (((size_t)head * o.pages.n + page_at(o.pages, b, s / kPage)) * kPage + s % kPage) * 128;
        return (((size_t)b * o.g + head) * o.cap + s) * 128;
    }
    __device__ __forceinline__ size_t v_at(int b, int head, int n, int s) const {
        if (o.pages.pt)
            return (((size_t)head * o.pages.n + page_at(o.pages, b, s / kPage)) * 128 + n) * kPage + s % kPage;
        return (((size_t)b * o.g + head) * 128 + n) * o.cap + s;
    }
    // Region of the wave's 128 columns: 0 = Q, 1 = K, 2 = V, -1 = past N.
    __device__ __forceinline__ int region(int nw, int N, int* head) const {
        if (nw >= N) return -1;
        if (nw < o.n_q) { *head = nw >> 7; return 0; }
        if (nw < o.n_q + o.n_kv) { *head = (nw - o.n_q) >> 7; return 1; }
        *head = (nw - o.n_q - o.n_kv) >> 7;
        return 2;
    }
    __device__ __forceinline__ void stage(int pass, f32x16 (&acc)[4][4], int mw, int nw, int lane,
                                          int M, int N, char* st) const {
        int head;
        const int reg = region(nw, N, &head);
        if (reg < 0) return;
        const int l32 = lane & 31, hi = lane >> 5;
        if (reg == 2) {
            if (pass != 0) return;
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4)
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb) {
                        const int n = 32 * nb + l32, u = 8 * mb + 2 * r4 + hi;
                        u32x2 v;
                        v[0] = pack2bf(acc[mb][nb][4 * r4 + 0], acc[mb][nb][4 * r4 + 1]);
                        v[1] = pack2bf(acc[mb][nb][4 * r4 + 2], acc[mb][nb][4 * r4 + 3]);
                        *(u32x2*)(st + n * 256 + ((u ^ (n & 31)) * 8)) = v;
                    }
            return;
        }
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = 32 * mb + 8 * (i >> 2) + 4 * hi + (i & 3);
                st_f32(st, m, l32, pass == 0 ? acc[mb][0][i] : acc[mb][1][i]);
                st_f32(st, m, 32 + l32, pass == 0 ? acc[mb][2][i] : acc[mb][3][i]);
            }
    }
    // Item t of the lane: staging row (lane + 64 t) / 4, rotation pairs 8 ((lane + 64 t) % 4) ..
    // + 7 of the pass's 32.
    __device__ __forceinline__ void prefetch(int pass, int mw, int nw, int lane, int M, int N,
                                             Pre& pre) const {
        int head;
        const int reg = region(nw, N, &head);
        if (reg != 0 && reg != 1) return;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int id = lane + 64 * t;
            const int m = min(mw + (id >> 2), M - 1);
            const int c0 = 32 * pass + 8 * (id & 3);
            const u32x4* tab = (const u32x4*)(o.rope + (size_t)(m % o.S) * 64 + c0);
#pragma unroll
            for (int q = 0; q < 4; ++q) pre.cs[t][q] = tab[q];
        }
    }
    __device__ __forceinline__ void flush(int pass, int mw, int nw, int lane, int M, int N,
                                          const char* st, const Pre& pre) const {
        int head;
        const int reg = region(nw, N, &head);
        if (reg < 0) return;
        if (reg == 2) {
            if (pass != 0) return;
            // V^T rows: 16 lanes x 16 bytes = one 128-position row n.
            const bool fast = (o.S % 8) == 0;
#pragma unroll 4
            for (int it = 0; it < 32; ++it) {
                const int n = 4 * it + (lane >> 4), k = lane & 15;   // chunk k = positions 8k..8k+7
                const int m = mw + 8 * k;
                if (m >= M) continue;
                const int sw = n & 31;
                const u32x2 lo = *(const u32x2*)(st + n * 256 + (((2 * k) ^ sw) * 8));
                const u32x2 up = *(const u32x2*)(st + n * 256 + (((2 * k + 1) ^ sw) * 8));
                const int b = m / o.S, s = m - b * o.S;
                if (fast && m + 7 < M) {
                    // s % 8 == 0: the 8 positions never straddle a 64-position page.
                    *(u32x4*)(o.vc + v_at(b, head, n, s)) = u32x4{lo[0], lo[1], up[0], up[1]};
                } else {
                    const uint32_t w4[4] = {lo[0], lo[1], up[0], up[1]};
                    for (int e = 0; e < 8 && m + e < M; ++e) {
                        int bb = b, ss = s + e;
                        while (ss >= o.S) { ss -= o.S; ++bb; }
                        o.vc[v_at(bb, head, n, ss)] = (bf16_t)(w4[e >> 1] >> (16 * (e & 1)));
                    }
                }
            }
            return;
        }
        // Q / K: 128 rows x 4 groups of 8 rotation pairs; 8 items per lane (cos/sin rows from
        // prefetch()).
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int id = lane + 64 * t, k = id & 3, rowl = id >> 2;
            const int m = mw + rowl;
            if (m >= M) continue;
            const u32x4 a0 = ld_f32(st, rowl, 2 * k), a1 = ld_f32(st, rowl, 2 * k + 1);
            const u32x4 b0 = ld_f32(st, rowl, 8 + 2 * k), b1 = ld_f32(st, rowl, 9 + 2 * k);
            float x1[8], x2[8], c[8], sn[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x1[e] = __uint_as_float(a0[e]);
                x1[e + 4] = __uint_as_float(a1[e]);
                x2[e] = __uint_as_float(b0[e]);
                x2[e + 4] = __uint_as_float(b1[e]);
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                c[e] = __uint_as_float(pre.cs[t][e >> 1][2 * (e & 1)]);
                sn[e] = __uint_as_float(pre.cs[t][e >> 1][2 * (e & 1) + 1]);
            }
            u32x4 lo, up;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                lo[e] = pack2bf(x1[2 * e] * c[2 * e] - x2[2 * e] * sn[2 * e],
                                x1[2 * e + 1] * c[2 * e + 1] - x2[2 * e + 1] * sn[2 * e + 1]);
                up[e] = pack2bf(x2[2 * e] * c[2 * e] + x1[2 * e] * sn[2 * e],
                                x2[2 * e + 1] * c[2 * e + 1] + x1[2 * e + 1] * sn[2 * e + 1]);
            }
            const int c0 = 32 * pass + 8 * k;
            uint16_t* dst;
            if (reg == 0) {
                dst = o.q + (size_t)m * o.n_q + head * 128;
            } else {
                const int b = m / o.S;
                dst = o.kc + k_row(b, head, m - b * o.S);
            }
            *(u32x4*)(dst + c0) = lo;
            *(u32x4*)(dst + c0 + 64) = up;
        }
    }
};

// Residual update y = x + acc.  x is the bf16 layer input (XF32 = false) or the fp32
// residual stream (XF32 = true, updated in place through yf); y is written in bf16,
// yf (optional) in fp32.  The fp32 tile is staged in two passes of 64 columns
// (128 x 64 fp32 = 32 KB per wave in 256-byte rows).
template <bool XF32>
struct ResidEpi {
    static constexpr int kPasses = 2;
    // The lane's 16 residual items (row, 8 columns), requested before the tile is staged.
    struct Pre {
        u32x4 xv[16][XF32 ? 2 : 1];
    };
    const void* x;
    uint16_t* y;
    float* yf;
    __device__ __forceinline__ void set_split(int) {}
    __device__ __forceinline__ void stage(int pass, f32x16 (&acc)[4][4], int mw, int nw, int lane,
                                          int M, int N, char* st) const {
        if (nw >= N) return;
        const int l32 = lane & 31, hi = lane >> 5;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = 32 * mb + 8 * (i >> 2) + 4 * hi + (i & 3);
                st_f32(st, m, l32, pass == 0 ? acc[mb][0][i] : acc[mb][2][i]);
                st_f32(st, m, 32 + l32, pass == 0 ? acc[mb][1][i] : acc[mb][3][i]);
            }
    }
    // Item it of the lane: row 8 it + lane / 8, columns 8 (lane % 8) .. + 7 of the pass's 64.
    __device__ __forceinline__ void prefetch(int pass, int mw, int nw, int lane, int M, int N,
                                             Pre& pre) const {
        if (nw >= N) return;
#pragma unroll
        for (int it = 0; it < 16; ++it) {
            const int ml = 8 * it + (lane >> 3), c8 = lane & 7;
            const size_t off = (size_t)min(mw + ml, M - 1) * N + nw + 64 * pass + 8 * c8;
            if (XF32) {
                pre.xv[it][0] = *(const u32x4*)((const float*)x + off);
                pre.xv[it][XF32 ? 1 : 0] = *(const u32x4*)((const float*)x + off + 4);
            } else {
                pre.xv[it][0] = *(const u32x4*)((const uint16_t*)x + off);
            }
        }
    }
    __device__ __forceinline__ void flush(int pass, int mw, int nw, int lane, int M, int N,
                                          const char* st, const Pre& pre) const {
        if (nw >= N) return;
        const auto& xv = pre.xv;
#pragma unroll
        for (int it = 0; it < 16; ++it) {
            const int ml = 8 * it + (lane >> 3), c8 = lane & 7;
            const int m = mw + ml;
            if (m >= M) continue;
            const u32x4 p0 = ld_f32(st, ml, 2 * c8), p1 = ld_f32(st, ml, 2 * c8 + 1);
            float r[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float a0 = __uint_as_float(p0[e]), a1 = __uint_as_float(p1[e]);
                float x0, x1;
                if (XF32) {
                    x0 = __uint_as_float(xv[it][0][e]);
                    x1 = __uint_as_float(xv[it][XF32 ? 1 : 0][e]);
                } else {
                    const uint32_t w0 = xv[it][0][e >> 1], w1 = xv[it][0][2 + (e >> 1)];
                    x0 = __uint_as_float((e & 1) ? (w0 & 0xFFFF0000u) : (w0 << 16));
                    x1 = __uint_as_float((e & 1) ? (w1 & 0xFFFF0000u) : (w1 << 16));
                }
                r[e] = x0 + a0;
                r[4 + e] = x1 + a1;
            }
            const size_t off = (size_t)m * N + nw + 64 * pass + 8 * c8;
            u32x4 out;
#pragma unroll
            for (int e = 0; e < 4; ++e) out[e] = pack2bf(r[2 * e], r[2 * e + 1]);
            *(u32x4*)(y + off) = out;
            if (yf) {
                *(u32x4*)(yf + off) = u32x4{__float_as_uint(r[0]), __float_as_uint(r[1]),
                                            __float_as_uint(r[2]), __float_as_uint(r[3])};
                *(u32x4*)(yf + off + 4) = u32x4{__float_as_uint(r[4]), __float_as_uint(r[5]),
                                                __float_as_uint(r[6]), __float_as_uint(r[7])};
            }
        }
    }
};

// Plain store of C (no fused work): bf16 [M][N], or fp32 partial sums of one K slice into
// plane `split` of out ([M][N] per plane).  Staged like ResidEpi, two passes of 64 columns.
struct OutEpi {
    static constexpr int kPasses = 2;
    struct Pre {};
    void* out;
    size_t plane;
    int split;
    bool bf16;
    __device__ __forceinline__ void set_split(int s) { split = s; }
    __device__ __forceinline__ void stage(int pass, f32x16 (&acc)[4][4], int mw, int nw, int lane,
                                          int M, int N, char* st) const {
        if (nw >= N) return;
        const int l32 = lane & 31, hi = lane >> 5;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = 32 * mb + 8 * (i >> 2) + 4 * hi + (i & 3);
                st_f32(st, m, l32, pass == 0 ? acc[mb][0][i] : acc[mb][2][i]);
                st_f32(st, m, 32 + l32, pass == 0 ? acc[mb][1][i] : acc[mb][3][i]);
            }
    }
    __device__ __forceinline__ void prefetch(int, int, int, int, int, int, Pre&) const {}
    __device__ __forceinline__ void flush(int pass, int mw, int nw, int lane, int M, int N,
                                          const char* st, const Pre&) const {
        if (nw >= N) return;
#pragma unroll
        for (int it = 0; it < 16; ++it) {
            const int ml = 8 * it + (lane >> 3), c8 = lane & 7;
            const int m = mw + ml;
            if (m >= M) continue;
            const u32x4 p0 = ld_f32(st, ml, 2 * c8), p1 = ld_f32(st, ml, 2 * c8 + 1);
            const size_t off = (size_t)m * N + nw + 64 * pass + 8 * c8;
            if (bf16) {
                u32x4 o;
                o[0] = pack2bf(__uint_as_float(p0[0]), __uint_as_float(p0[1]));
                o[1] = pack2bf(__uint_as_float(p0[2]), __uint_as_float(p0[3]));
                o[2] = pack2bf(__uint_as_float(p1[0]), __uint_as_float(p1[1]));
                o[3] = pack2bf(__uint_as_float(p1[2]), __uint_as_float(p1[3]));
                *(u32x4*)((uint16_t*)out + off) = o;
            } else {
                float* dst = (float*)out + split * plane + off;
                *(u32x4*)dst = p0;
                *(u32x4*)(dst + 4) = p1;
            }
        }
    }
};

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

// LDS position of 16-byte chunk c of tile row r (rows are 128 B): spreads 16 consecutive
// rows of one chunk column over all 64 banks.
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r >> 1) & 7); }

// BUF: operand tiles are fetched with buffer loads into LDS, each lane's 8 + 8 offsets
// computed once and the k-tile advance given as the scalar offset, so issuing a tile costs
// no vector instructions (operands below 2 GiB; a wave's 64 W rows lie in one weight block
// since block sizes and N are multiples of 128).
template <class Epi, bool BUF>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_nt(const uint16_t* __restrict__ A, WRows W,
                                                     int M, int N, int K, int splits, Epi epi) {
    __shared__ u32x4 lds[2][2][BM * 8];  // [stage][A, W][row * 8 + swizzled chunk]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN;
    // With split K, workgroup slot `split` of every tile takes K columns
    // [split * K / splits, (split + 1) * K / splits); consecutive ids share a slice.
    const int lid0 = xcd_remap(blockIdx.x, gridDim.x);
    const int split = lid0 / (ntm * ntn);
    const int lid = lid0 - split * (ntm * ntn);
    const int kofs = split * (K / splits);
    epi.set_split(split);
    const int group = lid / (GROUP_M * ntn), first = group * GROUP_M;
    const int gsz = min(ntm - first, GROUP_M);
    const int in_g = lid - group * GROUP_M * ntn;
    const int m0 = (first + in_g % gsz) * BM, n0 = (in_g / gsz) * BN;

    // Direct global -> LDS loads: wave w fills tile rows 64 w .. 64 w + 63 of A and of W,
    // eight 1 KB instructions each (8 rows of 128 B); lane l of instruction j covers row
    // 64 w + 8 j + l / 8 and fetches the global chunk that belongs at LDS position l % 8.
    const uint16_t* a_src[8];
    const uint16_t* w_src[8];
    uint32_t ga_off[8], gw_off[8];
    __amdgpu_buffer_rsrc_t ars, wrs;
    if constexpr (BUF) {
        const int wu = __builtin_amdgcn_readfirstlane(wave);
        ars = __builtin_amdgcn_make_buffer_rsrc((void*)A, 0, M * K * 2, kRsrcWord3);
        const int x = n0 + 64 * wu;              // tile row 64 w (past N if the wave has no real row)
        int nb = min(x, N - 1), blk = 0;
        if (nb >= W.rows[0]) {
            nb -= W.rows[0];
            blk = 1;
            if (nb >= W.rows[1]) {
                nb -= W.rows[1];
                blk = 2;
            }
        }
        const int rows_blk = W.rows[blk];
        wrs = __builtin_amdgcn_make_buffer_rsrc((void*)W.p[blk], 0, rows_blk * K * 2, kRsrcWord3);
        const int nrow0 = nb + (x - min(x, N - 1));   // block row of tile row 64 w (rows past the block clamp)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int row = 64 * wave + 8 * j + (lane >> 3);
            const int c = swz(row, lane & 7);
            ga_off[j] = (uint32_t)(min(m0 + row, M - 1) * K + kofs + 8 * c) * 2u;
            gw_off[j] = (uint32_t)(min(nrow0 + 8 * j + (lane >> 3), rows_blk - 1) * K + kofs + 8 * c) * 2u;
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int row = 64 * wave + 8 * j + (lane >> 3);
            const int c = swz(row, lane & 7);
            a_src[j] = A + (size_t)min(m0 + row, M - 1) * K + kofs + 8 * c;
            w_src[j] = w_row(W, min(n0 + row, N - 1), K) + kofs + 8 * c;
        }
    }
    // Row group j (8 rows of A and of W) of tile kt into stage stg.
    auto issue_part = [&](int kt, int stg, int j) {
        const int r0 = 64 * (BUF ? __builtin_amdgcn_readfirstlane(wave) : wave) + 8 * j;
        if constexpr (BUF) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ars, (lvoid_t*)&lds[stg][0][r0 * 8], 16, ga_off[j], kt * BK * 2,
                                                     0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lvoid_t*)&lds[stg][1][r0 * 8], 16, gw_off[j], kt * BK * 2,
                                                     0, 0);
        } else {
            __builtin_amdgcn_global_load_lds((gvoid_t*)(a_src[j] + kt * BK), (lvoid_t*)&lds[stg][0][r0 * 8], 16,
                                             0, 0);
            __builtin_amdgcn_global_load_lds((gvoid_t*)(w_src[j] + kt * BK), (lvoid_t*)&lds[stg][1][r0 * 8], 16,
                                             0, 0);
        }
    };
    auto issue = [&](int kt, int stg) {
#pragma unroll
        for (int j = 0; j < 8; ++j) issue_part(kt, stg, j);
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

    const int nk = K / splits / BK;
    const int l32 = lane & 31, hi = lane >> 5;
    int a_off[4], b_off[4], rsw[4], bsw[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int ra = wm * 128 + 32 * i + l32, rb = wn * 128 + 32 * i + l32;
        a_off[i] = ra * 8;
        b_off[i] = rb * 8;
        rsw[i] = (ra >> 1) & 7;
        bsw[i] = (rb >> 1) & 7;
    }
    auto load_frags = [&](int stg, int ks, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
        const int c = 2 * ks + hi;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            fa[i] = as_bf16x8(lds[stg][0][a_off[i] + (c ^ rsw[i])]);
            fb[i] = as_bf16x8(lds[stg][1][b_off[i] + (c ^ bsw[i])]);
        }
    };

    issue(0, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    bf16x8 fa[4], fb[4], ga[4], gb[4];
    load_frags(0, 0, fa, fb);
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < nk;
        // Four 16-wide k steps; the fragments of step ks + 1 are read from LDS while the
        // 16 MFMAs of step ks run (one ds_read slotted after each of the first 8 MFMAs).
        // Tile kt + 1 goes into the other buffer (last read before the barrier that ended
        // step kt - 1) in two halves, with the first two k steps: issued in one burst its
        // LDS writes collide with the fragment reads; spread over all four steps the last
        // loads land too close to the end-of-tile wait (measured: 4 % / 5 % faster GEMMs
        // than the burst at K = 2048 / 8192).
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            if (more && ks < 2) {
#pragma unroll
                for (int j = 0; j < 4; ++j) issue_part(kt + 1, cur ^ 1, 4 * ks + j);
            }
            if (ks < 3) load_frags(cur, ks + 1, ga, gb);
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = mfma32x32x16(fa[mb], fb[nb], acc[mb][nb]);
            if (ks < 3) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // 1 MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // 1 LDS read
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    fa[i] = ga[i];
                    fb[i] = gb[i];
                }
            }
        }
        if (more) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's part of tile kt + 1
            __syncthreads();                                    // everyone's part, and tile kt read
            load_frags(cur ^ 1, 0, fa, fb);
        }
    }
    // Epilogue through LDS, in Epi::kPasses passes over the wave's 32 KB.  The pass's global
    // inputs (cos/sin rows, residual) are requested before the staging, so that their latency
    // runs under the LDS writes and the barrier.
    char* st = (char*)&lds[0][0][0] + wave * 32768;
#pragma unroll
    for (int pass = 0; pass < Epi::kPasses; ++pass) {
        __syncthreads();   // the LDS is free: last fragment reads / previous flush are done
        typename Epi::Pre pre;
        epi.prefetch(pass, m0 + wm * 128, n0 + wn * 128, lane, M, N, pre);
        epi.stage(pass, acc, m0 + wm * 128, n0 + wn * 128, lane, M, N, st);
        __syncthreads();
        epi.flush(pass, m0 + wm * 128, n0 + wn * 128, lane, M, N, st, pre);
    }
}

// ---------------------------------------------------------------------------
// The same tiling for C[M][N] = sum_k A[k][m] B[k][n] with both operands given K-major
// ([K][rows], rows contiguous): the weight gradients dW_O = G^T O and
// dW_QKV = [dQ|dK|dV]^T X of the backward, whose K is the token axis.  Each operand tile is
// staged as [64 k][256 rows] in the sub-tiled layout and its MFMA fragments are taken along
// the tile's rows with the LDS transpose read (two ds_read_b64_tr_b16 each), so neither
// operand is copied transposed.  Any K: the last tile reads clamped rows, and the A
// fragments zero the rows past K.  (For products with K-major weights, dO = G W_O and
// dX += [dQ|dK|dV] W_stack, the row-major kernel on once-transposed weights is faster: the
// transpose read moves 8 bytes per lane per instruction against 16.)
// ---------------------------------------------------------------------------
// A K-major operand: k-rows of `ld` values, stacked from up to three buffers (p[i] holds
// rows[i] k-rows).  Written this way (templated operand, if-constexpr'd loads) the kernel
// compiles to 384 registers without spills; a plain single-pointer spelling of the same
// loop was compiled to 512 registers plus 130-180 spilled ones, 2.6x slower.
template <bool T>
struct Operand {
    WRows w;
    int ld;
    __device__ __forceinline__ const uint16_t* krow(int k) const {
        if (k < w.rows[0]) return (const uint16_t*)w.p[0] + (size_t)k * ld;
        k -= w.rows[0];
        if (k < w.rows[1]) return (const uint16_t*)w.p[1] + (size_t)k * ld;
        k -= w.rows[1];
        return (const uint16_t*)w.p[2] + (size_t)k * ld;
    }
};

template <class Epi, bool TA, bool TB>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_g(Operand<TA> Aop, Operand<TB> Bop, int M, int N, int K,
                                                    int splits, Epi epi) {
    __shared__ u32x4 lds[2][2][BM * 8];  // [stage][A, B]: [64 k][256] bf16, sub-tiled
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, hi = lane >> 5;
    const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN;
    const int lid0 = xcd_remap(blockIdx.x, gridDim.x);
    const int split = lid0 / (ntm * ntn);
    const int lid = lid0 - split * (ntm * ntn);
    epi.set_split(split);
    const int group = lid / (GROUP_M * ntn), first = group * GROUP_M;
    const int gsz = min(ntm - first, GROUP_M);
    const int in_g = lid - group * GROUP_M * ntn;
    const int m0 = (first + in_g % gsz) * BM, n0 = (in_g / gsz) * BN;
    const int nkt = (K + BK - 1) / BK;
    const int kt0 = split * nkt / splits, kt1 = (split + 1) * nkt / splits;
    const int ch = sub_chunk(lane);
    auto tsrc = [&](const auto& op, int c0, int C, int kt, int j) {
        const int u = 8 * wave + j, sb = u >> 2, q = u & 3;
        const int k = min(kt * BK + 16 * q + (lane >> 2), K - 1);
        const int col = min(c0 + 32 * sb + 8 * ch, C - 8);
        return op.krow(k) + col;
    };
    auto issue_part = [&](int kt, int stg, int j) {
        if constexpr (TA) {
            const int u = 8 * wave + j;
            __builtin_amdgcn_global_load_lds((gvoid_t*)tsrc(Aop, m0, M, kt, j),
                                             (lvoid_t*)((char*)&lds[stg][0][0] + (u >> 2) * 4096 + (u & 3) * 1024),
                                             16, 0, 0);
        }
        if constexpr (TB) {
            const int u = 8 * wave + j;
            __builtin_amdgcn_global_load_lds((gvoid_t*)tsrc(Bop, n0, N, kt, j),
                                             (lvoid_t*)((char*)&lds[stg][1][0] + (u >> 2) * 4096 + (u & 3) * 1024),
                                             16, 0, 0);
        }
    };
    auto issue = [&](int kt, int stg) {
#pragma unroll
        for (int j = 0; j < 8; ++j) issue_part(kt, stg, j);
    };
    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
    const bool ktail = TA && (K % BK) != 0;
    auto load_frags = [&](int stg, int kt, int ks, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (TA) fa[i] = tr_frag<BK, false>(lds[stg][0], 16 * ks, wm * 128 + 32 * i, lane);
            if constexpr (TB) fb[i] = tr_frag<BK, false>(lds[stg][1], 16 * ks, wn * 128 + 32 * i, lane);
        }
        if (ktail && kt == nkt - 1) {
            const int kb = kt * BK + 16 * ks + 8 * hi;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                u32x4 v = __builtin_bit_cast(u32x4, fa[i]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] &= (kb + 2 * e < K ? 0x0000FFFFu : 0u) | (kb + 2 * e + 1 < K ? 0xFFFF0000u : 0u);
                fa[i] = __builtin_bit_cast(bf16x8, v);
            }
        }
    };
    (void)l32;
    if (kt0 < kt1) {
        issue(kt0, 0);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        bf16x8 fa[4], fb[4], ga[4], gb[4];
        load_frags(0, kt0, 0, fa, fb);
        for (int kt = kt0; kt < kt1; ++kt) {
            const int cur = (kt - kt0) & 1;
            const bool more = kt + 1 < kt1;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                if (more && ks < 2) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) issue_part(kt + 1, cur ^ 1, 4 * ks + j);
                }
                if (ks < 3) load_frags(cur, kt, ks + 1, ga, gb);
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                    for (int nb2 = 0; nb2 < 4; ++nb2) acc[mb][nb2] = mfma32x32x16(fa[mb], fb[nb2], acc[mb][nb2]);
                if (ks < 3) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        fa[i] = ga[i];
                        fb[i] = gb[i];
                    }
                }
            }
            if (more) {
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                __syncthreads();
                load_frags(cur ^ 1, kt + 1, 0, fa, fb);
            }
        }
    }
    char* st = (char*)&lds[0][0][0] + wave * 32768;
#pragma unroll
    for (int pass = 0; pass < Epi::kPasses; ++pass) {
        __syncthreads();
        typename Epi::Pre pre;
        epi.prefetch(pass, m0 + wm * 128, n0 + wn * 128, lane, M, N, pre);
        epi.stage(pass, acc, m0 + wm * 128, n0 + wn * 128, lane, M, N, st);
        __syncthreads();
        epi.flush(pass, m0 + wm * 128, n0 + wn * 128, lane, M, N, st, pre);
    }
}

template <class Epi>
hipError_t launch(const uint16_t* A, const WRows& W, int M, int N, int K, const Epi& epi,
                  hipStream_t st, int splits = 1) {
    const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    bool buf = (int64_t)M * K * 2 < ((int64_t)1 << 31) && N % 128 == 0;
    for (int i = 0; i < 3; ++i) buf = buf && (int64_t)W.rows[i] * K * 2 < ((int64_t)1 << 31) && W.rows[i] % 128 == 0;
    if (buf)
        hipLaunchKernelGGL((gemm_bf16_nt<Epi, true>), dim3(tiles * splits), dim3(NT), 0, st, A, W, M, N, K, splits,
                           epi);
    else
        hipLaunchKernelGGL((gemm_bf16_nt<Epi, false>), dim3(tiles * splits), dim3(NT), 0, st, A, W, M, N, K,
                           splits, epi);
    return hipGetLastError();
}

}  // namespace

hipError_t gemm_qkv_bf16(const uint16_t* x, const WRows& w, int M, int N, int K, const QkvOut& o,
                         hipStream_t st) {
    return launch(x, w, M, N, K, QkvEpi{o}, st);
}

hipError_t gemm_resid_bf16(const uint16_t* a, const uint16_t* w, const void* x_res, bool x_f32,
                           uint16_t* y, float* yf, int M, int N, int K, hipStream_t st) {
    WRows W{{w, nullptr, nullptr}, {N, 0, 0}};
    if (x_f32) return launch(a, W, M, N, K, ResidEpi<true>{x_res, y, yf}, st);
    return launch(a, W, M, N, K, ResidEpi<false>{x_res, y, yf}, st);
}

hipError_t gemm_kmajor_out_bf16(const uint16_t* a, int lda, const uint16_t* b, int ldb, int M, int N, int K,
                                int splits, float* part, hipStream_t st) {
    if (splits < 1 || splits > (K + BK - 1) / BK || M % 8 || N % 8 || lda % 8 || ldb % 8)
        return hipErrorInvalidValue;
    Operand<true> A{{{a, nullptr, nullptr}, {K, 0, 0}}, lda};
    Operand<true> B{{{b, nullptr, nullptr}, {K, 0, 0}}, ldb};
    const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_bf16_g<OutEpi, true, true>), dim3(tiles * splits), dim3(NT), 0, st, A, B, M, N, K,
                       splits, OutEpi{part, (size_t)M * N, 0, false});
    return hipGetLastError();
}

hipError_t gemm_out_bf16(const uint16_t* a, const uint16_t* w, int M, int N, int K, uint16_t* c,
                         hipStream_t st) {
    if (K % BK) return hipErrorInvalidValue;
    WRows W{{w, nullptr, nullptr}, {N, 0, 0}};
    return launch(a, W, M, N, K, OutEpi{c, 0, 0, true}, st);
}

hipError_t gemm_nt_out_splits(const uint16_t* a, const uint16_t* w, int M, int N, int K, int splits, float* part,
                              hipStream_t st) {
    if (splits < 1 || K % (BK * splits)) return hipErrorInvalidValue;
    WRows W{{w, nullptr, nullptr}, {N, 0, 0}};
    return launch(a, W, M, N, K, OutEpi{part, (size_t)M * N, 0, false}, st, splits);
}

int gemm_out_splits(int M, int N, int K) {
    const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    const int nkt = (K + BK - 1) / BK;
    int s = 1;
    // One workgroup per CU: split K until the grid covers the 256 CUs (at most 8 slices, each
    // at least one 64-wide tile).
    while (tiles * s < 256 && 2 * s <= 8 && 2 * s <= nkt) s *= 2;
    return s;
}

}  // namespace kvp
