// Single-token decode attention over a long KV cache (Sec. 2.2: each new token
// attends to every cached position; a consumer reads its producer's cache,
// Eq. 3), split along the cache ("split-K") and merged by a second kernel.
//
// One wave = one split of one (sequence b, KV head): it streams positions
// [sp * split, min((sp + 1) * split, len_b + 1)) of the K and V^T slots straight
// from HBM into registers (no LDS: every byte is used once) and keeps an
// online softmax for the r query heads that share the KV head.
//
// Per 64-position tile: S^T[16 pos x 16 heads] blocks via
// v_mfma_f32_16x16x32_bf16 with A = K rows and B = Q^T (heads padded to 16),
// then O^T[128 x 16] += V^T P^T.  The MFMA row -> position assignment is
// permuted so that after the score MFMAs each lane holds 8 consecutive
// positions of its head, which is exactly the k-slice the PV MFMA needs and a
// 16-byte run of the V^T row: K is read as 64-byte row segments and V^T as
// 64-byte row segments, P never leaves registers.  The next tile's loads are
// issued before the current tile is consumed.
//
// The partial results (running max m, sum l, unnormalised O) of every split go
// to a workspace; decode_combine merges them per (b, head).
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

constexpr int D = 128, TILE = 64, NT = 256, PSTRIDE = D + 4;  // O[128], m, l, pad
constexpr float kLazy = 8.0f;

struct DTile {
    u32x4 k[4][4];   // [block tb][k step ks]
    u32x4 v[8][2];   // [d block db][pv step s]
};

__global__ __launch_bounds__(NT, 1) void decode_attn_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc, const uint16_t* __restrict__ Vc,
    const int32_t* __restrict__ lens, float* __restrict__ part, int B, int a, int g, int cap,
    int split, int nsplit, float scale_log2) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int sp = blockIdx.x * (NT / 64) + wave;
    const int kvh = blockIdx.y, b = blockIdx.z;
    const int r = a / g;
    // Positions [0, len_b] inclusive; clamping keeps every access inside the slot
    // even if a length exceeds what the host validated.
    const int len = max(0, min(lens[b], cap - 1)) + 1;
    const int p_begin = sp * split;
    if (sp >= nsplit || p_begin >= len) return;
    const int p_end = min(p_begin + split, len);

    const int col = lane & 15, grp = lane >> 4;    // MFMA column (head) and lane group

    // Q^T fragments: lane (col, grp) holds head kvh*r + col, dims 32 ks + 8 grp + 0..7.
    bf16x8 qf[4];
    {
        const bool real = col < r;
        const uint16_t* qrow = Q + (size_t)b * a * D + (size_t)(kvh * r + (real ? col : 0)) * D + 8 * grp;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            u32x4 v = *(const u32x4*)(qrow + 32 * ks);
            if (!real) v = u32x4{0, 0, 0, 0};
            qf[ks] = as_bf16x8(v);
        }
    }

    const uint16_t* kbase = Kc + ((size_t)b * g + kvh) * cap * D;
    const uint16_t* vbase = Vc + ((size_t)b * g + kvh) * D * cap;

    // Position held by MFMA row rho (= lane & 15 for the A operand) of score block tb
    // of a tile: block 2s + e covers positions 32 s + 8 (rho / 4) + 4 e + rho % 4.
    auto load = [&](int t0, DTile& tl) {
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
            const int s = tb >> 1, e = tb & 1;
            const int pos = t0 + 32 * s + 8 * (col >> 2) + 4 * e + (col & 3);
            const uint16_t* kr = kbase + (size_t)pos * D + 8 * grp;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) tl.k[tb][ks] = *(const u32x4*)(kr + 32 * ks);
        }
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const uint16_t* vr = vbase + (size_t)(16 * db + col) * cap + t0 + 8 * grp;
#pragma unroll
            for (int s = 0; s < 2; ++s) tl.v[db][s] = *(const u32x4*)(vr + 32 * s);
        }
    };

    f32x4 o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = f32x4{};
    float m_run = -INFINITY, l_run = 0.f;

    // Tiles start on 64-position boundaries; cap % 64 == 0 keeps every load in the slot.
    const int t_first = p_begin & ~(TILE - 1);
    DTile cur, nxt;
    load(t_first, cur);
    for (int t0 = t_first; t0 < p_end; t0 += TILE) {
        const bool more = t0 + TILE < p_end;
        if (more) load(t0 + TILE, nxt);

        // ---- scores --------------------------------------------------------------
        f32x4 sc[4];
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
            sc[tb] = f32x4{};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) sc[tb] = mfma16x16x32(as_bf16x8(cur.k[tb][ks]), qf[ks], sc[tb]);
        }
        // Lane (col, grp) now holds head col at positions t0 + 32 s + 8 grp + 4 e + i.
        const bool edge = (t0 < p_begin) || (t0 + TILE > p_end);
        float mx = -INFINITY;
#pragma unroll
        for (int tb = 0; tb < 4; ++tb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (edge) {
                    const int pos = t0 + 32 * (tb >> 1) + 8 * grp + 4 * (tb & 1) + i;
                    if (pos < p_begin || pos >= p_end) sc[tb][i] = -INFINITY;
                }
                mx = fmaxf(mx, sc[tb][i]);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mt = mx * scale_log2;
        if (__any(mt > m_run + kLazy)) {
            const float m_new = fmaxf(m_run, mt);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < 8; ++db) o[db] *= alpha;
        }
        bf16x8 pb[2];
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            float p[8];
#pragma unroll
            for (int e = 0; e < 2; ++e)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    p[4 * e + i] = __builtin_amdgcn_exp2f(fmaf(sc[2 * s + e][i], scale_log2, -m_run));
                    l_run += p[4 * e + i];
                }
            u32x4 w;
            w[0] = pack2bf(p[0], p[1]);
            w[1] = pack2bf(p[2], p[3]);
            w[2] = pack2bf(p[4], p[5]);
            w[3] = pack2bf(p[6], p[7]);
            pb[s] = as_bf16x8(w);
        }
        // ---- O^T += V^T P^T; positions outside [p_begin, p_end) carry P = 0 but their V
        // must be finite: zero them (the cache beyond len_b may hold anything).
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int p0 = t0 + 32 * s + 8 * grp;
#pragma unroll
            for (int db = 0; db < 8; ++db) {
                u32x4 v = cur.v[db][s];
                if (edge) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int pa = p0 + 2 * e, pbn = pa + 1;
                        const uint32_t m = ((pa >= p_begin && pa < p_end) ? 0x0000FFFFu : 0u) |
                                           ((pbn >= p_begin && pbn < p_end) ? 0xFFFF0000u : 0u);
                        v[e] &= m;
                    }
                }
                o[db] = mfma16x16x32(as_bf16x8(v), pb[s], o[db]);
            }
        }
        if (more) cur = nxt;
    }

    // ---- partial result of this split ------------------------------------------------
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (col < r) {
        float* pr = part + (((size_t)b * a + kvh * r + col) * nsplit + sp) * PSTRIDE;
        // O^T block db: lane holds dims 16 db + 4 grp + 0..3 of head col.
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            *(f32x4*)(pr + 16 * db + 4 * grp) = o[db];
        }
        if (grp == 0) {
            pr[D] = m_run;
            pr[D + 1] = l_run;
        }
    }
}

__global__ __launch_bounds__(D) void decode_combine_kernel(const float* __restrict__ part,
                                                           const int32_t* __restrict__ lens,
                                                           uint16_t* __restrict__ O, int a, int cap,
                                                           int split, int nsplit) {
    const int bh = blockIdx.x, b = bh / a, d = threadIdx.x;
    const int len = max(0, min(lens[b], cap - 1)) + 1;
    const int nvalid = min(nsplit, (len + split - 1) / split);
    const float* pr = part + (size_t)bh * nsplit * PSTRIDE;
    float M = -INFINITY;
    for (int s = 0; s < nvalid; ++s) M = fmaxf(M, pr[(size_t)s * PSTRIDE + D]);
    float num = 0.f, den = 0.f;
    for (int s = 0; s < nvalid; ++s) {
        const float w = exp2f(pr[(size_t)s * PSTRIDE + D] - M);
        den += w * pr[(size_t)s * PSTRIDE + D + 1];
        num += w * pr[(size_t)s * PSTRIDE + d];
    }
    O[(size_t)bh * D + d] = f2bf(num / den);
}

}  // namespace

hipError_t decode_attn_bf16(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                            const int32_t* lens, float* part, int B, int a, int g, int cap,
                            int split, int nsplit, hipStream_t st) {
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    dim3 grid((nsplit + 3) / 4, g, B);
    hipLaunchKernelGGL(decode_attn_kernel, grid, dim3(NT), 0, st, q, kc, vc, lens, part, B, a, g, cap,
                       split, nsplit, scale_log2);
    return hipGetLastError();
}

hipError_t decode_combine_bf16(const float* part, const int32_t* lens, uint16_t* o, int B, int a,
                               int cap, int split, int nsplit, hipStream_t st) {
    hipLaunchKernelGGL(decode_combine_kernel, dim3(B * a), dim3(D), 0, st, part, lens, o, a, cap, split,
                       nsplit);
    return hipGetLastError();
}

}  // namespace kvp
