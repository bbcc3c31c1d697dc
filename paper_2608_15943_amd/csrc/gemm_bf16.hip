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
//   * residual: X_{l+1} = X_l + O W_O^T.
//
// Tiling: 256 x 256 x 64 per workgroup of 4 waves (2 x 2, 128 x 128 each, a
// 4 x 4 grid of 32 x 32 MFMA blocks = 256 fp32 accumulators per lane).
// Operand tiles go global -> registers -> LDS, double buffered (2 x 64 KB),
// one barrier per K step; LDS rows are 128 B with the 16-byte chunk index
// XOR-swizzled by (row & 7) so that the 32-row fragment reads spread over all
// banks.  Tiles are ordered so that each XCD works on a contiguous group of
// M-panels (its own L2 keeps the A and W panels hot).
#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

constexpr int BM = 256, BN = 256, BK = 64, NT = 256, GROUP_M = 8;

__device__ __forceinline__ const uint16_t* w_row(const WRows& w, int n, int K) {
    if (n < w.rows[0]) return (const uint16_t*)w.p[0] + (size_t)n * K;
    n -= w.rows[0];
    if (n < w.rows[1]) return (const uint16_t*)w.p[1] + (size_t)n * K;
    n -= w.rows[1];
    return (const uint16_t*)w.p[2] + (size_t)n * K;
}

struct QkvEpi {
    QkvOut o;
    __device__ __forceinline__ void operator()(f32x16 (&acc)[4][4], int mw, int nw, int lane, int M,
                                               int N) const {
        if (nw >= N) return;
        const int l32 = lane & 31, hi = lane >> 5;
        if (nw >= o.n_q + o.n_kv) {
            // V (not rotated), stored transposed: four consecutive rows of a lane are
            // four consecutive positions, one 8-byte store when they share a sequence.
            const int head = (nw - o.n_q - o.n_kv) >> 7;
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const int mrow0 = mw + 32 * mb + 8 * r4 + 4 * hi;
                    if (mrow0 >= M) continue;
                    const int b0 = mrow0 / o.S, s0 = mrow0 - b0 * o.S;
                    const bool packed = (mrow0 + 3 < M) && (s0 + 3 < o.S) && ((s0 & 3) == 0) &&
                                        ((o.cap & 3) == 0);
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb) {
                        const int c = 32 * nb + l32;
                        if (packed) {
                            u32x2 v;
                            v.x = pack2bf(acc[mb][nb][4 * r4 + 0], acc[mb][nb][4 * r4 + 1]);
                            v.y = pack2bf(acc[mb][nb][4 * r4 + 2], acc[mb][nb][4 * r4 + 3]);
                            *(u32x2*)(o.vc + (((size_t)b0 * o.g + head) * 128 + c) * o.cap + s0) = v;
                        } else {
                            for (int r = 0; r < 4 && mrow0 + r < M; ++r) {
                                int b = b0, s = s0 + r;
                                while (s >= o.S) {  // 4 rows can span several sequences when S < 4
                                    s -= o.S;
                                    ++b;
                                }
                                o.vc[(((size_t)b * o.g + head) * 128 + c) * o.cap + s] =
                                    f2bf(acc[mb][nb][4 * r4 + r]);
                            }
                        }
                    }
                }
            return;
        }
        // Q or K: rotate the pair (c, c + 64) of each head by the position's angle.
        const bool is_q = nw < o.n_q;
        const int head = is_q ? (nw >> 7) : ((nw - o.n_q) >> 7);
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int mrow0 = mw + 32 * mb + 8 * r4 + 4 * hi;
                const int b0 = mrow0 / o.S, s0 = mrow0 - b0 * o.S;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = mrow0 + r;
                    if (m >= M) break;
                    int b = b0, s = s0 + r;
                    while (s >= o.S) {  // 4 rows can span several sequences when S < 4
                        s -= o.S;
                        ++b;
                    }
                    uint16_t* dst = is_q ? o.q + (size_t)m * o.n_q + head * 128
                                         : o.kc + (((size_t)b * o.g + head) * o.cap + s) * 128;
#pragma unroll
                    for (int nb = 0; nb < 2; ++nb) {
                        const int c = 32 * nb + l32;
                        const float2 cs = o.rope[(size_t)s * 64 + c];
                        const float x1 = acc[mb][nb][4 * r4 + r], x2 = acc[mb][nb + 2][4 * r4 + r];
                        dst[c] = f2bf(x1 * cs.x - x2 * cs.y);
                        dst[c + 64] = f2bf(x2 * cs.x + x1 * cs.y);
                    }
                }
            }
    }
};

struct ResidEpi {
    const uint16_t* x;
    uint16_t* y;
    __device__ __forceinline__ void operator()(f32x16 (&acc)[4][4], int mw, int nw, int lane, int M,
                                               int N) const {
        const int l32 = lane & 31, hi = lane >> 5;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = mw + 32 * mb + 8 * (i >> 2) + 4 * hi + (i & 3);
                if (m >= M) continue;
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) {
                    const int n = nw + 32 * nb + l32;
                    if (n < N) {
                        const size_t off = (size_t)m * N + n;
                        y[off] = f2bf(bf2f(x[off]) + acc[mb][nb][i]);
                    }
                }
            }
    }
};

template <class Epi>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_nt(const uint16_t* __restrict__ A, WRows W,
                                                     int M, int N, int K, Epi epi) {
    __shared__ u32x4 lds[2][2][BM * 8];  // [stage][A, W][row * 8 + swizzled chunk]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN;
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int group = lid / (GROUP_M * ntn), first = group * GROUP_M;
    const int gsz = min(ntm - first, GROUP_M);
    const int in_g = lid - group * GROUP_M * ntn;
    const int m0 = (first + in_g % gsz) * BM, n0 = (in_g / gsz) * BN;

    // Loader: thread covers rows (tid >> 3) + 32 i of both tiles, 16-byte chunk tid & 7.
    const int kc = tid & 7;
    const u32x4* a_src[8];
    const u32x4* w_src[8];
    int soff[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int row = (tid >> 3) + 32 * i;
        a_src[i] = (const u32x4*)(A + (size_t)min(m0 + row, M - 1) * K) + kc;
        w_src[i] = (const u32x4*)w_row(W, min(n0 + row, N - 1), K) + kc;
        soff[i] = row * 8 + (kc ^ (row & 7));
    }

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

    u32x4 ra[8], rw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        ra[i] = a_src[i][0];
        rw[i] = w_src[i][0];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        lds[0][0][soff[i]] = ra[i];
        lds[0][1][soff[i]] = rw[i];
    }
    __syncthreads();

    const int nk = K / BK;
    const int l32 = lane & 31, hi = lane >> 5;
    // LDS offsets (in 16-byte chunks) of this lane's fragment rows; row & 7 == l32 & 7.
    int a_off[4], b_off[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a_off[i] = (wm * 128 + 32 * i + l32) * 8;
        b_off[i] = (wn * 128 + 32 * i + l32) * 8;
    }
    const int sw = l32 & 7;
    auto load_frags = [&](int stg, int ks, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
        const int c = (2 * ks + hi) ^ sw;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            fa[i] = as_bf16x8(lds[stg][0][a_off[i] + c]);
            fb[i] = as_bf16x8(lds[stg][1][b_off[i] + c]);
        }
    };

    bf16x8 fa[4], fb[4], ga[4], gb[4];
    load_frags(0, 0, fa, fb);
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                ra[i] = a_src[i][(kt + 1) * 8];
                rw[i] = w_src[i][(kt + 1) * 8];
            }
        }
        // Four 16-wide k steps; the fragments of step ks + 1 are read from LDS while the
        // 16 MFMAs of step ks run (one ds_read slotted after each of the first 8 MFMAs).
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
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
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                lds[cur ^ 1][0][soff[i]] = ra[i];
                lds[cur ^ 1][1][soff[i]] = rw[i];
            }
        }
        __syncthreads();
        if (more) load_frags(cur ^ 1, 0, fa, fb);
    }
    epi(acc, m0 + wm * 128, n0 + wn * 128, lane, M, N);
}

template <class Epi>
hipError_t launch(const uint16_t* A, const WRows& W, int M, int N, int K, const Epi& epi,
                  hipStream_t st) {
    const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    hipLaunchKernelGGL(gemm_bf16_nt<Epi>, dim3(tiles), dim3(NT), 0, st, A, W, M, N, K, epi);
    return hipGetLastError();
}

}  // namespace

hipError_t gemm_qkv_bf16(const uint16_t* x, const WRows& w, int M, int N, int K, const QkvOut& o,
                         hipStream_t st) {
    return launch(x, w, M, N, K, QkvEpi{o}, st);
}

hipError_t gemm_resid_bf16(const uint16_t* a, const uint16_t* w, const uint16_t* x_res,
                           uint16_t* y, int M, int N, int K, hipStream_t st) {
    WRows W{{w, nullptr, nullptr}, {N, 0, 0}};
    return launch(a, W, M, N, K, ResidEpi{x_res, y}, st);
}

}  // namespace kvp
