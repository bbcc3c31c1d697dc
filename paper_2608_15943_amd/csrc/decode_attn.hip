// Single-token decode attention over a long KV cache (Sec. 2.2: each new token
// attends to every cached position; a consumer reads its producer's cache,
// Eq. 3), split along the cache ("split-K") and merged by a second kernel.
//
// Schedule: the work of one layer is the list of 64-position tiles of every
// (sequence b, KV head) pair, in (b, head, tile) order.  The grid has one wave per
// SIMD of the device, all resident at once, and wave w streams the contiguous
// range [w c, (w + 1) c) of that list with c = ceil(tiles / waves): every wave
// reads the same number of bytes whatever the mix of lengths, and a range may run
// from the end of one pair into the next without a pipeline bubble.  Each piece
// of a range that lies in one pair ends in a partial result (running max m, sum
// l, unnormalised O); the piece of wave w in pair P goes to slot w + P, which is
// unique because w and P never both decrease along the list.
//
// Per tile: S^T[16 pos x 16 heads] blocks via v_mfma_f32_16x16x32_bf16 with
// A = K rows and B = Q^T (the r query heads of the KV head, padded to 16), then
// O^T[128 x 16] += V^T P^T.  The MFMA row -> position assignment is permuted so
// that after the score MFMAs each lane holds 8 consecutive positions of its
// head, which is exactly the k-slice the PV MFMA needs and a 16-byte run of the
// V^T row: K and V^T are read as 64-byte row segments straight from HBM into
// registers (no LDS: every byte is used once) and P never leaves registers.  The
// next tile's loads (and the next pair's queries) are issued before the current
// tile is consumed.

#include <math.h>

#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

constexpr int D = 128, TILE = 64, PSTRIDE = D + 4;  // O[128], m, l, pad
constexpr int kCombineThreads = 256;
constexpr float kLazy = 8.0f;

struct DTile {
    u32x4 k[4][4];   // [block tb][k step ks]
    u32x4 v[8][2];   // [d block db][pv step s]
};

// Tiles of every sequence (lanes < B) and their inclusive prefix over sequences.
struct SeqTiles {
    int len, n, pre;
};

__device__ __forceinline__ SeqTiles seq_tiles(const int32_t* lens, int B, int cap, int lane) {
    SeqTiles t;
    t.len = lane < B ? max(0, min(lens[lane], cap - 1)) + 1 : 0;
    t.n = (t.len + TILE - 1) / TILE;
    t.pre = t.n;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(t.pre, off);
        if (lane >= off) t.pre += v;
    }
    return t;
}

// One wave per workgroup, one workgroup per SIMD (the grid is sized to the device).
// PAGED: every 64-position tile is one page, looked up once per tile.
template <bool PAGED>
__global__ __launch_bounds__(64, 1) void decode_attn_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc, const uint16_t* __restrict__ Vc,
    const int32_t* __restrict__ lens, float* __restrict__ part, int B, int a, int g, int cap,
    float scale_log2, Pages pages) {
    const int lane = threadIdx.x;
    const int W = gridDim.x, w = blockIdx.x;
    const int r = a / g;
    const SeqTiles st = seq_tiles(lens, B, cap, lane);
    const long long T = (long long)g * __shfl(st.pre, 63);
    const long long c = (T + W - 1) / W;
    long long x = (long long)w * c;
    const long long x_end = min(x + c, T);
    if (x >= x_end) return;

    // Locate tile x: sequence b is the number of sequences that end at or before x.
    int b = __popcll(__ballot((long long)g * st.pre <= x));
    int n = __shfl(st.n, b), len = __shfl(st.len, b);
    const long long rem = x - (long long)g * (__shfl(st.pre, b) - n);
    int kvh = (int)(rem / n), t = (int)(rem % n);

    const int col = lane & 15, grp = lane >> 4;    // MFMA column (head) and lane group

    // Q^T fragments: lane (col, grp) holds head kvh*r + col, dims 32 ks + 8 grp + 0..7.
    auto load_q = [&](int qb, int qh, bf16x8* qf) {
        const bool real = col < r;
        const uint16_t* qrow = Q + (size_t)qb * a * D + (size_t)(qh * r + (real ? col : 0)) * D + 8 * grp;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            u32x4 v = *(const u32x4*)(qrow + 32 * ks);
            if (!real) v = u32x4{0, 0, 0, 0};
            qf[ks] = as_bf16x8(v);
        }
    };

    // Position held by MFMA row rho (= lane & 15 for the A operand) of score block tb
    // of a tile: block 2s + e covers positions 32 s + 8 (rho / 4) + 4 e + rho % 4.
    // Tiles start at multiples of 64 and cap % 64 == 0, so every load stays in the slot
    // (or, paged, in the tile's page).  Paged: the wave keeps 64 consecutive entries of a
    // table row in a register (lane i: entry 64 c + i of row pb) and reads the tile's entry
    // with readlane, so a dependent table load is paid once per 64 tiles, not per tile.
    int pb = -1, pc = -1, pgv = 0;
    auto load = [&](int lb, int lh, int t0, DTile& tl) {
        const uint16_t* kbase;
        const uint16_t* vbase;
        int vld;
        if constexpr (PAGED) {
            const int j = t0 / TILE;
            if (lb != pb || (j >> 6) != pc) {
                pb = lb;
                pc = j >> 6;
                const int e = 64 * pc + lane;
                pgv = e < pages.stride ? pages.pt[(size_t)lb * pages.stride + e] : 0;
            }
            const int pg = min(max(__builtin_amdgcn_readlane(pgv, j & 63), 0), pages.n - 1);
            kbase = Kc + ((size_t)lh * pages.n + pg) * TILE * D - (size_t)t0 * D;
            vbase = Vc + ((size_t)lh * pages.n + pg) * D * TILE - t0;
            vld = TILE;
        } else {
            kbase = Kc + ((size_t)lb * g + lh) * cap * D;
            vbase = Vc + ((size_t)lb * g + lh) * D * cap;
            vld = cap;
        }
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
            const uint16_t* vr = vbase + (size_t)(16 * db + col) * vld + t0 + 8 * grp;
#pragma unroll
            for (int s = 0; s < 2; ++s) tl.v[db][s] = *(const u32x4*)(vr + 32 * s);
        }
    };

    bf16x8 qf[4], qn[4];
    load_q(b, kvh, qf);
    f32x4 o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = f32x4{};
    float m_run = -INFINITY, l_run = 0.f;

    DTile cur, nxt;
    load(b, kvh, TILE * t, cur);
    for (; x < x_end; ++x) {
        // Next tile of the range, possibly in the next pair.
        const bool more = x + 1 < x_end;
        int nb = b, nh = kvh, nt = t + 1, nn = n, nl = len;
        bool pair_ends = !more;
        if (more) {
            if (nt == n) {
                nt = 0;
                pair_ends = true;
                if (++nh == g) {
                    nh = 0;
                    ++nb;
                    nn = __shfl(st.n, nb);
                    nl = __shfl(st.len, nb);
                }
                load_q(nb, nh, qn);
            }
            load(nb, nh, TILE * nt, nxt);
        }

        // ---- scores --------------------------------------------------------------
        const int t0 = TILE * t;
        f32x4 sc[4];
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
            sc[tb] = f32x4{};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) sc[tb] = mfma16x16x32(as_bf16x8(cur.k[tb][ks]), qf[ks], sc[tb]);
        }
        // Lane (col, grp) now holds head col at positions t0 + 32 s + 8 grp + 4 e + i.
        const bool edge = t0 + TILE > len;
        float mx = -INFINITY;
#pragma unroll
        for (int tb = 0; tb < 4; ++tb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (edge) {
                    const int pos = t0 + 32 * (tb >> 1) + 8 * grp + 4 * (tb & 1) + i;
                    if (pos >= len) sc[tb][i] = -INFINITY;
                }
                mx = fmaxf(mx, sc[tb][i]);
            }
        mx = pair32_max(pair16_max(mx));
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
            u32x4 wv;
            wv[0] = pack2bf(p[0], p[1]);
            wv[1] = pack2bf(p[2], p[3]);
            wv[2] = pack2bf(p[4], p[5]);
            wv[3] = pack2bf(p[6], p[7]);
            pb[s] = as_bf16x8(wv);
        }
        // ---- O^T += V^T P^T; positions >= len carry P = 0 but their V must be finite:
        // zero them (the cache beyond len_b may hold anything).
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int p0 = t0 + 32 * s + 8 * grp;
#pragma unroll
            for (int db = 0; db < 8; ++db) {
                u32x4 v = cur.v[db][s];
                if (edge) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int pa = p0 + 2 * e;
                        const uint32_t m = (pa < len ? 0x0000FFFFu : 0u) | (pa + 1 < len ? 0xFFFF0000u : 0u);
                        v[e] &= m;
                    }
                }
                o[db] = mfma16x16x32(as_bf16x8(v), pb[s], o[db]);
            }
        }

        if (pair_ends) {
            // ---- partial result of this wave's piece of pair (b, kvh) -----------------
            const float lt = pair32_sum(pair16_sum(l_run));
            if (col < r) {
                float* pr = part + (((size_t)w + (size_t)b * g + kvh) * r + col) * PSTRIDE;
                // O^T block db: lane holds dims 16 db + 4 grp + 0..3 of head col.
#pragma unroll
                for (int db = 0; db < 8; ++db) *(f32x4*)(pr + 16 * db + 4 * grp) = o[db];
                if (grp == 0) {
                    pr[D] = m_run;
                    pr[D + 1] = lt;
                }
            }
            if (more) {
#pragma unroll
                for (int i = 0; i < 8; ++i) o[i] = f32x4{};
                m_run = -INFINITY;
                l_run = 0.f;
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) qf[ks] = qn[ks];
            }
        }
        b = nb;
        kvh = nh;
        t = nt;
        n = nn;
        len = nl;
        if (more) cur = nxt;
    }
}

// Merge the pieces of one (sequence, query head): the waves that covered its pair are
// w_first..w_last (recomputed from the lengths exactly as the attention kernel splits
// the tile list).  Weights 2^(m_s - M) go to LDS, then each half of the block sums
// every other piece for its 128 dimensions (coalesced 512-byte rows, independent
// loads), so the merge costs a few load latencies rather than one per piece.
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(
    const float* __restrict__ part, const int32_t* __restrict__ lens, uint16_t* __restrict__ O, int B,
    int a, int g, int cap, int W) {
    __shared__ float wsh[kMaxDecodeSplits];
    __shared__ float red[2][kCombineThreads / 64];
    __shared__ float half1[D];
    const int bh = blockIdx.x, b = bh / a, j = bh % a, t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int r = a / g, kvh = j / r, jr = j % r;
    const SeqTiles st = seq_tiles(lens, B, cap, lane);
    const long long T = (long long)g * __shfl(st.pre, 63);
    const long long c = (T + W - 1) / W;
    const int n = __shfl(st.n, b);
    const long long g0 = (long long)g * (__shfl(st.pre, b) - n) + (long long)kvh * n;
    const int w_first = (int)(g0 / c), w_last = (int)((g0 + n - 1) / c);
    const int ns = w_last - w_first + 1;
    const float* pr = part + (((size_t)w_first + (size_t)b * g + kvh) * r + jr) * PSTRIDE;
    const size_t step = (size_t)r * PSTRIDE;     // next wave's slot for the same pair
    float M = -INFINITY;
    for (int s = t; s < ns; s += kCombineThreads) M = fmaxf(M, pr[s * step + D]);
    M = wave_max(M);
    if (lane == 0) red[0][wave] = M;
    __syncthreads();
    M = red[0][0];
#pragma unroll
    for (int v = 1; v < kCombineThreads / 64; ++v) M = fmaxf(M, red[0][v]);
    float den = 0.f;
    for (int s = t; s < ns; s += kCombineThreads) {
        const float wt = exp2f(pr[s * step + D] - M);
        wsh[s] = wt;
        den += wt * pr[s * step + D + 1];
    }
    den = wave_sum(den);
    if (lane == 0) red[1][wave] = den;
    __syncthreads();
    den = 0.f;
#pragma unroll
    for (int v = 0; v < kCombineThreads / 64; ++v) den += red[1][v];
    const int d = t & (D - 1), hf = t / D;
    float num = 0.f;
#pragma unroll 8
    for (int s = hf; s < ns; s += 2) num += wsh[s] * pr[s * step + d];
    if (hf == 1) half1[d] = num;
    __syncthreads();
    if (hf == 0) O[(size_t)bh * D + d] = f2bf((num + half1[d]) / den);
}

}  // namespace

hipError_t decode_attn_bf16(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                            const int32_t* lens, float* part, int B, int a, int g, int cap, int waves,
                            const Pages& pages, hipStream_t st) {
    if (B < 1 || B > 64 || waves < 1 || waves > kMaxDecodeSplits) return hipErrorInvalidValue;
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    if (pages.pt) {
        if (pages.n < 1 || pages.stride < 1 || cap != TILE * pages.stride) return hipErrorInvalidValue;
        hipLaunchKernelGGL(decode_attn_kernel<true>, dim3(waves), dim3(64), 0, st, q, kc, vc, lens, part, B, a,
                           g, cap, scale_log2, pages);
    } else {
        hipLaunchKernelGGL(decode_attn_kernel<false>, dim3(waves), dim3(64), 0, st, q, kc, vc, lens, part, B,
                           a, g, cap, scale_log2, pages);
    }
    return hipGetLastError();
}

hipError_t decode_combine_bf16(const float* part, const int32_t* lens, uint16_t* o, int B, int a, int g,
                               int cap, int waves, hipStream_t st) {
    if (B < 1 || B > 64 || waves < 1 || waves > kMaxDecodeSplits) return hipErrorInvalidValue;
    hipLaunchKernelGGL(decode_combine_kernel, dim3(B * a), dim3(kCombineThreads), 0, st, part, lens, o, B,
                       a, g, cap, waves);
    return hipGetLastError();
}

}  // namespace kvp
